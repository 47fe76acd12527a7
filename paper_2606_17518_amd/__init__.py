"""MI355X (gfx950) fork-decode attention, KV-block import/export and per-step
append for SpecGen's speculative forks (arXiv 2606.17518): a HIP library
behind a C ABI (include/specgen.h) and its Python binding."""
from .binding import (EXPORTED, ForkBatchTensors, SpecgenError, SPECGEN_BF16, SPECGEN_FLAG_FP8_SCORES, SPECGEN_FP32, SPECGEN_FP8_E4M3,
                      SPECGEN_PATH_AUTO, SPECGEN_PATH_DOT, SPECGEN_PATH_MFMA, SPECGEN_PHASE_ALL, SPECGEN_PHASE_MERGE,
                      SPECGEN_NOALLOC_SCRATCH_BYTES, SPECGEN_PHASE_PARTIALS, alloc_prefill_workspace, alloc_workspace, host_batch_struct, lib,
                      specgen_fork_decode_attn_phase, specgen_fork_prefill_attn,
                      specgen_fork_prefill_attn_workspace_size,
                      specgen_fork_decode_attn, specgen_fork_decode_attn_noalloc, specgen_fork_decode_attn_split, specgen_fork_decode_attn_workspace_size, specgen_kv_append,
                      specgen_kv_export, specgen_kv_import, specgen_lse_merge)
