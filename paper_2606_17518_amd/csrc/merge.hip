// merge.hip -- log-sum-exp merge of partial attention results.
//
// Partials over disjoint key sets combine exactly: with M = max_s lse_s and
// w_s = exp(lse_s - M), out = sum_s w_s o_s / sum_s w_s and
// lse = M + ln sum_s w_s (a part with lse = -inf is empty and is skipped).
// One wavefront merges one output row: lane p first takes part p's lse to
// find the running max and weights (chunks of 64 parts, rescaled between
// chunks), then all lanes sweep the parts over the head dimension.
#include <algorithm>

#include "merge.h"

namespace specgen {

// Merge `nparts` parts of one row.  part_o(p) -> const float* (row vector of
// D floats), part_lse(p) -> float.  Writes out (bf16 or fp32) and lse.
template <int VEC, typename PO, typename PL>
__device__ __forceinline__ void merge_row(int nparts, int D, PO part_o, PL part_lse, void* out_row,
                                          bool out_bf16, float* out_lse_p) {
  const int lane = threadIdx.x & 63;
  float M = -INFINITY, z = 0.f;
  float acc[VEC];
#pragma unroll
  for (int v = 0; v < VEC; ++v) acc[v] = 0.f;
  for (int p0 = 0; p0 < nparts; p0 += 64) {
    const int p = p0 + lane;
    const float l = p < nparts ? part_lse(p) : -INFINITY;
    float cm = l;
    for (int o = 32; o >= 1; o >>= 1) cm = fmaxf(cm, __shfl_xor(cm, o, 64));
    const float Mn = fmaxf(M, cm);
    if (Mn == -INFINITY) continue;   // every part so far empty
    const float rescale = __expf(M - Mn);   // M = -inf -> 0
    z *= rescale;
#pragma unroll
    for (int v = 0; v < VEC; ++v) acc[v] *= rescale;
    M = Mn;
    const float wl = (l == -INFINITY) ? 0.f : __expf(l - M);
    float zs = wl;
    for (int o = 32; o >= 1; o >>= 1) zs += __shfl_xor(zs, o, 64);
    z += zs;
    const int cnt = (nparts - p0) < 64 ? (nparts - p0) : 64;
    for (int q = 0; q < cnt; ++q) {
      const float wq = __shfl(wl, q, 64);
      if (wq == 0.f) continue;   // wave-uniform
      const float* o = part_o(p0 + q);
#pragma unroll
      for (int v = 0; v < VEC; ++v) {
        const int d = lane + 64 * v;
        if (d < D) acc[v] = fmaf(wq, o[d], acc[v]);
      }
    }
  }
  const bool empty = (M == -INFINITY);
  const float inv = empty ? 0.f : 1.f / z;
#pragma unroll
  for (int v = 0; v < VEC; ++v) {
    const int d = lane + 64 * v;
    if (d < D) {
      const float r = empty ? 0.f : acc[v] * inv;
      if (out_bf16) reinterpret_cast<uint16_t*>(out_row)[d] = f32_to_bf16(r);
      else reinterpret_cast<float*>(out_row)[d] = r;
    }
  }
  if (out_lse_p && lane == 0) *out_lse_p = empty ? -INFINITY : M + __logf(z);
}

// ---- standalone merge: o_parts [S][R][D], lse_parts [S][R] -------------------
template <int VEC>
__global__ void __launch_bounds__(256) lse_merge_kernel(const float* __restrict__ o_parts,
                                                        const float* __restrict__ lse_parts, int S,
                                                        int64_t R, int D, void* __restrict__ out,
                                                        int out_bf16, float* __restrict__ out_lse) {
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= R) return;
  auto po = [&](int p) { return o_parts + ((int64_t)p * R + r) * D; };
  auto pl = [&](int p) { return lse_parts[(int64_t)p * R + r]; };
  void* orow = out_bf16 ? (void*)(reinterpret_cast<uint16_t*>(out) + r * D)
                        : (void*)(reinterpret_cast<float*>(out) + r * D);
  merge_row<VEC>(S, D, po, pl, orow, out_bf16 != 0, out_lse ? out_lse + r : nullptr);
}

hipError_t launch_lse_merge(const float* o_parts, const float* lse_parts, int S, int64_t R, int D,
                            void* out, bool out_bf16, float* out_lse, hipStream_t stream) {
  if (R == 0) return hipSuccess;
  const dim3 grid((unsigned)((R + 3) / 4)), block(256);
  const int vec = (D + 63) / 64;
  switch (vec) {
#define SG_CASE(V) case V: hipLaunchKernelGGL(lse_merge_kernel<V>, grid, block, 0, stream, o_parts, lse_parts, S, R, D, out, (int)out_bf16, out_lse); break;
    SG_CASE(1) SG_CASE(2) SG_CASE(3) SG_CASE(4) SG_CASE(5) SG_CASE(6) SG_CASE(7) SG_CASE(8)
    SG_CASE(9) SG_CASE(10) SG_CASE(11) SG_CASE(12) SG_CASE(13) SG_CASE(14) SG_CASE(15) SG_CASE(16)
#undef SG_CASE
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// ---- fork merge: the parts of row (f, h) are the partials of the workers that
// covered its prefix items and its suffix item ---------------------------------

template <int D, int kDepth, int kU>
__global__ void __launch_bounds__(256) fork_merge_kernel(const Plan plan_arg, const float* __restrict__ ws, uint16_t* __restrict__ out,
                                                         float* __restrict__ out_lse) {
  __shared__ Plan splan;
  __shared__ MergeItemLoc sloc[4][kDepth + 1];   // each wave's item table (nested prefixes)
  plan_to_lds<256>(plan_arg, splan);
  // a wave per row; with more rows than the grid holds, waves take every
  // (4 * gridDim.x)-th row, so fewer workgroups copy the plan
  const int64_t rows = (int64_t)splan.N * splan.Hq;
  for (int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); row < rows; row += (int64_t)gridDim.x * 4)
    fork_merge_row<D, kDepth, kU>(splan, ws, row, out, out_lse, sloc[threadIdx.x >> 6]);
}

// Rows of at most kParts parts each, several rows per wave (merge.h).
template <int D, int kDepth, int kParts>
__global__ void __launch_bounds__(256) fork_merge_grouped_kernel(const Plan plan_arg, const float* __restrict__ ws,
                                                                 uint16_t* __restrict__ out, float* __restrict__ out_lse) {
  __shared__ Plan splan;
  plan_to_lds<256>(plan_arg, splan);
  constexpr int kRowsPerWave = 64 / (D / 8);
  const int64_t rows = (int64_t)splan.N * splan.Hq;
  const int grp = (threadIdx.x & 63) / (D / 8);
  for (int64_t r0 = ((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6)) * kRowsPerWave; r0 < rows;
       r0 += (int64_t)gridDim.x * 4 * kRowsPerWave)
    fork_merge_rows_grouped<D, kDepth, kParts>(splan, ws, r0 + grp, out, out_lse);
}

hipError_t launch_fork_merge(const Plan& plan, const float* ws, void* out, float* out_lse, hipStream_t stream) {
  const int64_t rows = (int64_t)plan.N * plan.Hq;
  constexpr int64_t kMaxMergeBlocks = 2048;   // 8 per CU; beyond that waves loop over rows
  const dim3 grid((unsigned)std::min<int64_t>((rows + 3) / 4, kMaxMergeBlocks)), block(256);
  // the merge walks as many prefix items per row as the longest chain needs,
  // rounded up to 1, 2, 4 or kMaxDepth
  const int dep = plan.depth <= 1 ? 1 : plan.depth <= 2 ? 2 : plan.depth <= 4 ? 4 : kMaxDepth;
  // parts per batch: the fewest load instructions per batch (2, 8 or all 64
  // parts) that cover every row of the plan in one batch.  A kernel holding 8
  // parts per batch needs about 60 registers, one holding 64 about 150, and a
  // compute unit holds correspondingly fewer waves of the larger one.
  const int ppi = 64 / (plan.D / 8);   // parts per load instruction
  const int mp = max_parts_per_row(plan);
  // Several rows per wave where every row has at most 16 parts (one batch), or
  // where there are so many rows that holding more of them in flight beats one
  // batch per row (a wave of the one-row layout holds one row, 3-7 waves per SIMD).
  if (dep <= 2 && (mp <= 16 || rows >= 8192)) {
    const int64_t per_block = 4 * (64 / (plan.D / 8));
    const dim3 g2((unsigned)std::min<int64_t>((rows + per_block - 1) / per_block, kMaxMergeBlocks));
    const int key = (plan.D == 128 ? 100 : 0) + dep * 10 + (mp <= 8 ? 8 : 16);
    switch (key) {
#define SG_GROUPED(DD, DEP, NP)                                                                          \
  case (DD == 128 ? 100 : 0) + DEP * 10 + NP:                                                              \
    hipLaunchKernelGGL((fork_merge_grouped_kernel<DD, DEP, NP>), g2, block, 0, stream, plan, ws,          \
                       (uint16_t*)out, out_lse);                                                         \
    break;
      SG_GROUPED(128, 1, 8) SG_GROUPED(128, 2, 8) SG_GROUPED(128, 1, 16) SG_GROUPED(128, 2, 16)
      SG_GROUPED(64, 1, 8) SG_GROUPED(64, 2, 8) SG_GROUPED(64, 1, 16) SG_GROUPED(64, 2, 16)
#undef SG_GROUPED
      default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
  }
  const int tier = mp <= 2 * ppi ? 1 : mp <= 8 * ppi ? 2 : 0;
  switch (dep * 1000 + plan.D + tier) {
#define SG_CASE(DEP, DD)                                                                                          \
  case DEP * 1000 + DD:                                                                                           \
    hipLaunchKernelGGL((fork_merge_kernel<DD, DEP, 64 / (64 / (DD / 8))>), grid, block, 0, stream, plan, ws,     \
                       (uint16_t*)out, out_lse);                                                                  \
    break;                                                                                                        \
  case DEP * 1000 + DD + 1:                                                                                       \
    hipLaunchKernelGGL((fork_merge_kernel<DD, DEP, 2>), grid, block, 0, stream, plan, ws, (uint16_t*)out, out_lse); \
    break;                                                                                                        \
  case DEP * 1000 + DD + 2:                                                                                       \
    hipLaunchKernelGGL((fork_merge_kernel<DD, DEP, 8>), grid, block, 0, stream, plan, ws, (uint16_t*)out, out_lse); \
    break;
    SG_CASE(1, 128) SG_CASE(2, 128) SG_CASE(4, 128) SG_CASE(kMaxDepth, 128)
    SG_CASE(1, 64) SG_CASE(2, 64) SG_CASE(4, 64) SG_CASE(kMaxDepth, 64)
#undef SG_CASE
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace specgen
