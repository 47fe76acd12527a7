// common.h -- device types and small helpers shared by the gfx950 kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace specgen {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

#define SG_LDS __attribute__((address_space(3)))

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// fp32 -> bf16 bits, round to nearest even (NaN stays NaN).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  __bf16 h = (__bf16)f;
  return __builtin_bit_cast(uint16_t, h);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return (uint32_t)f32_to_bf16(lo) | ((uint32_t)f32_to_bf16(hi) << 16);
}

__device__ __forceinline__ float wave_max_xor(float v, int mask) {
  return fmaxf(v, __shfl_xor(v, mask, 64));
}

__device__ __forceinline__ int uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }

// Partial-result and plan arguments shared by the attention kernels.
struct AttnArgs {
  const uint16_t* __restrict__ q;          // [N][Hq][D] bf16 bits
  const uint8_t* __restrict__ k_pool;      // [blocks][16][Hkv][D] kv elements
  const uint8_t* __restrict__ v_pool;
  const float* __restrict__ k_scale;       // [blocks] (E4M3 only)
  const float* __restrict__ v_scale;
  const int32_t* __restrict__ prefix_table_off;
  const int32_t* __restrict__ prefix_table;
  const int32_t* __restrict__ suffix_len;
  const int32_t* __restrict__ suffix_table_off;
  const int32_t* __restrict__ suffix_table;
  float* __restrict__ ws;                  // workspace (partials)
  float sm_scale;
  float c_log2;                            // sm_scale * log2(e)
};

}  // namespace specgen
