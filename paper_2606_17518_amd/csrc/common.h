// common.h -- device types and small helpers shared by the gfx950 kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "plan.h"

namespace specgen {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

#define SG_LDS __attribute__((address_space(3)))

constexpr float kLog2e = 1.4426950408889634f;

// fp32 -> bf16 bits, round to nearest even (NaN stays NaN).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  __bf16 h = (__bf16)f;
  return __builtin_bit_cast(uint16_t, h);
}

// Two fp32 -> packed bf16 pair (round to nearest even), one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const f32x2 v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

// Two fp32 -> packed fp16 pair (round to nearest even).
__device__ __forceinline__ uint32_t pack_f16x2(float lo, float hi) {
  typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
  const f32x2 v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, f16x2_t));
}

// Packed fp16 pair -> two fp32 (exact).
__device__ __forceinline__ f32x2 unpack_f16x2(uint32_t w) {
  typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
  return __builtin_convertvector(__builtin_bit_cast(f16x2_t, w), f32x2);
}

// Max / sum over the four 16-lane rows of a wave (lanes l, l^16, l^32, l^48)
// with the gfx950 row-swap permutes (no LDS round trip).
__device__ __forceinline__ float rows4_max(float v) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float rows4_sum(float v) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// Max / sum over the 16 lanes of each row with DPP moves (quad swaps, then
// the half-row and row mirrors): VALU work, no LDS round trip.
#define SG_DPP(v, ctrl) __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), (ctrl), 0xF, 0xF, false))
__device__ __forceinline__ float row16_max(float v) {
  v = fmaxf(v, SG_DPP(v, 0xB1));    // quad_perm [1,0,3,2]
  v = fmaxf(v, SG_DPP(v, 0x4E));    // quad_perm [2,3,0,1]
  v = fmaxf(v, SG_DPP(v, 0x141));   // row_half_mirror
  return fmaxf(v, SG_DPP(v, 0x140));   // row_mirror
}
__device__ __forceinline__ float row16_sum(float v) {
  v += SG_DPP(v, 0xB1);
  v += SG_DPP(v, 0x4E);
  v += SG_DPP(v, 0x141);
  return v + SG_DPP(v, 0x140);
}
// v + the value of lane l ^ 8 (rotation by 8 within the 16-lane row)
__device__ __forceinline__ float xor8_sum(float v) { return v + SG_DPP(v, 0x128); }

__device__ __forceinline__ int uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }

// Workgroup barrier for LDS hand-offs only: waits for this wave's LDS
// operations, then s_barrier.  Unlike __syncthreads() it does not wait for
// outstanding global loads (vector loads and stores share one counter on
// gfx950, so a workgroup release fence would drain the prefetched tiles).
// The memory clobber keeps the compiler from moving memory accesses across it.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// Wait for every outstanding vector-memory operation of this wave.  Used at
// the end of rarely taken paths that load registers the hot loop later reads,
// so the compiler does not place that wait inside the hot loop instead.
__device__ __forceinline__ void wait_vmem() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// LDS swizzle of K chunks: XOR-ed so a 16-key MFMA operand read hits
// distinct banks.
template <int CPR>
__device__ __forceinline__ int swz_k(int tok) { return ((tok & 3) | ((tok >> 1) & 12)) & (CPR - 1); }

// Partial-result and plan arguments shared by the attention kernels.
struct AttnArgs {
  const uint16_t* __restrict__ q;          // [N][Hq][D] bf16 bits
  const uint8_t* __restrict__ k_pool;      // [blocks][Hkv][16][D] kv elements
  // v_pool: [blocks][Hkv][D][16] (transposed)
  const uint8_t* __restrict__ v_pool;
  const float* __restrict__ k_scale;       // [blocks] (E4M3 only)
  const float* __restrict__ v_scale;
  const int32_t* __restrict__ prefix_table;
  const int32_t* __restrict__ suffix_table;
  float* __restrict__ ws;                  // workspace (partials)
  float sm_scale;
  float c_log2;                            // sm_scale * log2(e)
};

}  // namespace specgen
