// kernels.h -- host-side launchers of the device kernels (one per .hip file).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.h"
#include "plan.h"

namespace specgen {

// attn_bf16.hip (MFMA partition: bf16 or E4M3 KV)
hipError_t launch_attn_mfma_any(const AttnArgs& a, const Plan& plan, bool fp8, bool qk8, hipStream_t stream);
int mfma_tile_tokens(int D, bool fp8);
int mfma_item_cap();
int mfma_tile_cap(int D, bool fp8);
int mfma_walk_threads();
int mfma_rows();
// attn_dot.hip
hipError_t launch_attn_dot_any(const AttnArgs& a, const Plan& plan, bool fp8, hipStream_t stream);
int dot_tile_tokens(int D);
int dot_rows();
int dot_item_cap();
int dot_tile_cap(int D);
// merge.hip
hipError_t launch_fork_merge(const Plan& plan, const float* ws, void* out, float* out_lse, hipStream_t stream);
hipError_t launch_lse_merge(const float* o_parts, const float* lse_parts, int S, int64_t R, int D, void* out,
                            bool out_bf16, float* out_lse, hipStream_t stream);
// kv_import.hip: whole-block moves between the pool and a staging buffer
// (import: staging block i -> pool block ids[i]; export: the reverse)
struct BlockCopyTensor {
  uint8_t* pool;       // written by import, read by export
  uint8_t* staging;    // read by import, written by export
  int64_t block_bytes;
};
struct BlockCopyArgs {
  BlockCopyTensor t[4];
  int32_t num_tensors;
  const int32_t* ids;  // [n] pool block of each staging block
  int64_t n;
  int64_t num_pool_blocks;
  int32_t* bad_id_count;
};
hipError_t launch_kv_import(const BlockCopyArgs& a, hipStream_t stream);
hipError_t launch_kv_export(const BlockCopyArgs& a, hipStream_t stream);
// kv_append.hip: one new token per fork written into its suffix blocks
struct AppendArgs {
  uint8_t* k_pool;
  uint8_t* v_pool;
  const uint8_t* k_new;            // [N][Hkv][D] elements of elem_bytes
  const uint8_t* v_new;
  const int32_t* pos;              // [N]
  const int32_t* suffix_table_off; // [N+1]
  const int32_t* suffix_table;
  int32_t* bad_count;
  int64_t num_blocks;
  int32_t num_forks, num_kv_heads, head_dim, elem_bytes;
};
hipError_t launch_kv_append(const AppendArgs& a, hipStream_t stream);

}  // namespace specgen
