// abi.hip -- the extern "C" entry points declared in include/specgen.h:
// argument checks (all before any launch), the host planner that turns the
// host length mirrors into the work split of plan.h, and kernel dispatch.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <atomic>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/specgen.h"
#include "kernels.h"
#include "planner.h"
#include "table_check.h"


using namespace specgen;

namespace {

thread_local std::string g_last_error;

specgen_status_t fail(specgen_status_t st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

specgen_status_t ok() { return SPECGEN_OK; }

int device_cus() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  // per device, shared by every calling thread (each stores the same value)
  static std::atomic<int> cached[64];
  if (dev >= 0 && dev < 64) {
    const int c = cached[dev].load(std::memory_order_relaxed);
    if (c > 0) return c;
  }
  int cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0) cus = 256;
  if (dev >= 0 && dev < 64) cached[dev].store(cus, std::memory_order_relaxed);
  return cus;
}

// A block-table offset mirror off[0..n] for lengths len[0..n-1]: off[0] >= 0,
// and range i, [off[i], off[i+1]), holds at least ceil(len[i] / 16) ids.
specgen_status_t check_table_offsets(const char* what, const int32_t* off, const int32_t* len, int n) {
  if (n > kMaxForks) n = kMaxForks;   // the planner rejects larger batches
  if (off[0] < 0) return fail(SPECGEN_ERR_INVALID_ARG, "%s_table_off[0] = %d must be >= 0", what, off[0]);
  for (int i = 0; i < n; ++i) {
    if (off[i + 1] < off[i])
      return fail(SPECGEN_ERR_INVALID_ARG, "%s_table_off must be nondecreasing (index %d)", what, i);
    const int64_t need = len[i] > 0 ? ((int64_t)len[i] + kBlock - 1) / kBlock : 0;
    if ((int64_t)off[i + 1] - off[i] < need)
      return fail(SPECGEN_ERR_INVALID_ARG, "%s_table_off gives %d ids to entry %d, which needs %lld", what,
                  off[i + 1] - off[i], i, (long long)need);
  }
  return ok();
}

// Checks the batch and builds the plan; `ws_floats` receives the workspace size.
// `ptab_sel` (internal, [T] or NULL): traces whose prefix ids index the suffix table.
specgen_status_t build_plan(const specgen_fork_batch_t* b, Plan* plan, int64_t* ws_floats,
                            const int32_t* ptab_sel = nullptr) {
  if (!b) return fail(SPECGEN_ERR_INVALID_ARG, "batch is NULL");
  if (b->flags & ~SPECGEN_FLAG_FP8_SCORES) return fail(SPECGEN_ERR_INVALID_ARG, "unknown flags 0x%x", b->flags);
  if (b->num_traces < 1) return fail(SPECGEN_ERR_INVALID_ARG, "num_traces must be >= 1 (got %d)", b->num_traces);
  if (b->num_forks < 1) return fail(SPECGEN_ERR_INVALID_ARG, "num_forks must be >= 1 (got %d)", b->num_forks);
  if (b->block_size != 16) return fail(SPECGEN_ERR_UNSUPPORTED, "block_size %d must be 16", b->block_size);
  if (b->num_blocks < 1) return fail(SPECGEN_ERR_INVALID_ARG, "num_blocks must be >= 1");
  if (!(b->sm_scale > 0.f) || !std::isfinite(b->sm_scale))
    return fail(SPECGEN_ERR_INVALID_ARG, "sm_scale must be finite and > 0");
  if (b->kv_dtype != SPECGEN_BF16 && b->kv_dtype != SPECGEN_FP8_E4M3)
    return fail(SPECGEN_ERR_UNSUPPORTED, "kv_dtype %d not supported", b->kv_dtype);
  if (b->path != SPECGEN_PATH_AUTO && b->path != SPECGEN_PATH_DOT && b->path != SPECGEN_PATH_MFMA)
    return fail(SPECGEN_ERR_INVALID_ARG, "path %d unknown", b->path);
  if (!b->q || !b->k_pool || !b->v_pool || !b->fork_off || !b->prefix_len || !b->prefix_table_off ||
      !b->prefix_table || !b->suffix_len || !b->suffix_table_off)
    return fail(SPECGEN_ERR_INVALID_ARG, "a device pointer of the batch is NULL");
  if ((b->flags & SPECGEN_FLAG_FP8_SCORES) && b->kv_dtype != SPECGEN_FP8_E4M3)
    return fail(SPECGEN_ERR_INVALID_ARG, "fp8 scores need E4M3 KV");
  if ((b->flags & SPECGEN_FLAG_FP8_SCORES) && b->head_dim != 128)
    return fail(SPECGEN_ERR_UNSUPPORTED, "fp8 scores need head_dim 128");
  if (b->kv_dtype == SPECGEN_FP8_E4M3 && (!b->k_scale || !b->v_scale))
    return fail(SPECGEN_ERR_INVALID_ARG, "E4M3 KV needs k_scale and v_scale");
  if (!b->fork_off_h || !b->prefix_len_h || !b->suffix_len_h || !b->prefix_table_off_h || !b->suffix_table_off_h)
    return fail(SPECGEN_ERR_INVALID_ARG, "a host mirror of the batch is NULL");
  if (!b->suffix_table) {   // only a batch without suffix tokens may omit the suffix table
    for (int f = 0; f < b->num_forks; ++f)
      if (b->suffix_len_h[f] > 0) return fail(SPECGEN_ERR_INVALID_ARG, "suffix_table is NULL but fork %d has suffix tokens", f);
  }
  if (!ptab_sel) {
    // The caller's table offsets: non-negative, nondecreasing, and each range
    // long enough for its length (the kernels read ceil(len/16) ids from the
    // start of a range, with no bound of their own).  Internal batches
    // (ptab_sel set) derive their offsets from a batch checked here.
    specgen_status_t st = check_table_offsets("prefix", b->prefix_table_off_h, b->prefix_len_h, b->num_traces);
    if (st != SPECGEN_OK) return st;
    st = check_table_offsets("suffix", b->suffix_table_off_h, b->suffix_len_h, b->num_forks);
    if (st != SPECGEN_OK) return st;
  }
  const bool fp8 = b->kv_dtype == SPECGEN_FP8_E4M3;
  PlanInputs in;
  in.T = b->num_traces;
  in.N = b->num_forks;
  in.Hq = b->num_q_heads;
  in.Hkv = b->num_kv_heads;
  in.D = b->head_dim;
  in.policy = b->path;
  in.fork_off = b->fork_off_h;
  in.prefix_parent = b->prefix_parent_h;
  in.prefix_in_suffix_table = ptab_sel;
  in.prefix_len = b->prefix_len_h;
  in.suffix_len = b->suffix_len_h;
  in.prefix_table_off = b->prefix_table_off_h;
  in.suffix_table_off = b->suffix_table_off_h;
  in.tt[0] = mfma_tile_tokens(in.D == 64 ? 64 : 128, fp8);
  in.tt[1] = dot_tile_tokens(in.D);
  in.rbs[0] = mfma_rows();
  in.rbs[1] = dot_rows();
  in.item_cap[0] = mfma_item_cap();
  in.item_cap[1] = dot_item_cap();
  in.tile_cap[0] = mfma_tile_cap(in.D == 64 ? 64 : 128, fp8);
  in.tile_cap[1] = dot_tile_cap(in.D);
  // Unit prices of the split, from per-worker timelines of the MFMA kernel on
  // MI355X, in eighths of a tile of an item of 4 groups of 32 rows.  bf16 KV: a
  // tile of 1 or 4 groups took 1.20 and 1.32-1.36 us, and a prefix item's
  // fixed cost (its q slot, about 1 us, and its end: token-group combine and
  // partial stores, about 2.5 us) about 2.5 such tiles; the prefix-item charge
  // is 20 (workers whose range holds two items ended last at a charge of 16).
  // A suffix item (g rows) ends with far less to combine and store: at a charge
  // of 20 the workers holding suffix items ended 2.5-3 us before the others on
  // the 32k-prefix workload, at 12 with them.  E4M3 KV (which adds
  // the decode of each tile): 1.56-1.60, 1.96 and 2.96 us for 1, 4 and 8
  // groups, charge 16.  Items of 5-8 groups run one token group per wave
  // (each wave takes both 32-token slabs of a tile).  The dot path prices
  // every tile alike and an item at one tile.
  const int mfma_rg_bf16[9] = {0, 7, 7, 7, 8, 10, 11, 12, 13};
  const int mfma_rg_e4m3[9] = {0, 6, 6, 7, 8, 9, 10, 10, 11};
  for (int r = 0; r < 9; ++r) {
    in.wt_rg[0][r] = fp8 ? mfma_rg_e4m3[r] : mfma_rg_bf16[r];
    in.wt_rg[1][r] = 1;
  }
  in.charge[0] = fp8 ? 16 : 20;
  in.charge[1] = 1;
  in.charge_suf[0] = fp8 ? 16 : 12;
  in.charge_suf[1] = 1;
  in.walk_threads[0] = mfma_walk_threads();
  in.walk_threads[1] = 0;   // the dot kernel walks serially
  char err[256];
  const int rc = plan_build(in, [] { return device_cus(); }, plan, ws_floats, err, sizeof err);
  if (rc == kPlanInvalid) return fail(SPECGEN_ERR_INVALID_ARG, "%s", err);
  if (rc == kPlanUnsupported) return fail(SPECGEN_ERR_UNSUPPORTED, "%s", err);
  return ok();
}

#ifdef SPECGEN_DEBUG_CHECKS
// The debug build's check of every block id the partial kernels will read
// (table_check.h): the read part of each block table is copied to the host
// on `stream`, which is then synchronised, before anything is launched.
specgen_status_t debug_check_block_ids(const specgen_fork_batch_t* b, const Plan& plan, hipStream_t stream) {
  auto fetch = [&](int table, int64_t first, int64_t count, int32_t* dst) {
    const int32_t* src = table == 0 ? b->prefix_table : b->suffix_table;
    if (!src) return false;
    return hipMemcpyAsync(dst, src + first, (size_t)count * sizeof(int32_t), hipMemcpyDeviceToHost, stream) ==
               hipSuccess &&
           hipStreamSynchronize(stream) == hipSuccess;
  };
  BadBlockId bad;
  const int rc = check_block_ids(plan, b->num_blocks, fetch, &bad);
  if (rc == kTableFetchFailed) return fail(SPECGEN_ERR_DEVICE, "debug check: the block tables could not be read back");
  if (rc == kTableBadId)
    return fail(SPECGEN_ERR_INVALID_ARG, "debug check: %s_table[%lld] = %d, read by %s %d, is outside [0, %lld)",
                bad.table == 0 ? "prefix" : "suffix", (long long)bad.entry, bad.id,
                bad.kind == 0 ? "the prefix of trace" : "the suffix of fork", bad.owner, (long long)b->num_blocks);
  return ok();
}
#endif

// Queues one call of the split attention (both phases or one) for a checked
// batch and its plan.
specgen_status_t run_plan(const specgen_fork_batch_t* b, const Plan& plan, int64_t wsf, int32_t phase, void* out,
                          float* out_lse, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (!out && phase != SPECGEN_PHASE_PARTIALS) return fail(SPECGEN_ERR_INVALID_ARG, "out is NULL");
  if ((size_t)(wsf * 4) > workspace_bytes || (wsf > 0 && !workspace))
    return fail(SPECGEN_ERR_WORKSPACE, "workspace of %zu bytes, need %lld", workspace_bytes, (long long)(wsf * 4));
  if (((uintptr_t)workspace & 255) != 0) return fail(SPECGEN_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
  if (((uintptr_t)b->q & 15) || ((uintptr_t)b->k_pool & 15) || ((uintptr_t)b->v_pool & 15))
    return fail(SPECGEN_ERR_INVALID_ARG, "q, k_pool and v_pool must be 16-byte aligned");
  AttnArgs a;
  a.q = static_cast<const uint16_t*>(b->q);
  a.k_pool = static_cast<const uint8_t*>(b->k_pool);
  a.v_pool = static_cast<const uint8_t*>(b->v_pool);
  a.k_scale = b->k_scale;
  a.v_scale = b->v_scale;
  a.prefix_table = b->prefix_table;
  a.suffix_table = b->suffix_table;
  a.ws = static_cast<float*>(workspace);
  a.sm_scale = b->sm_scale;
  a.c_log2 = b->sm_scale * kLog2e;
  const bool fp8 = b->kv_dtype == SPECGEN_FP8_E4M3;
#ifdef SPECGEN_DEBUG_CHECKS
  if (phase != SPECGEN_PHASE_MERGE) {
    const specgen_status_t st = debug_check_block_ids(b, plan, stream);
    if (st != SPECGEN_OK) return st;
  }
#endif
  hipError_t e = hipSuccess;
  if (phase != SPECGEN_PHASE_MERGE) {
    const bool qk8 = (b->flags & SPECGEN_FLAG_FP8_SCORES) != 0;
    if (plan.part[kPartMfma].workers > 0) e = launch_attn_mfma_any(a, plan, fp8, qk8, stream);
    if (e == hipSuccess && plan.part[kPartDot].workers > 0) e = launch_attn_dot_any(a, plan, fp8, stream);
  }
  if (e == hipSuccess && phase != SPECGEN_PHASE_PARTIALS) e = launch_fork_merge(plan, a.ws, out, out_lse, stream);
  if (e != hipSuccess) return fail(SPECGEN_ERR_DEVICE, "kernel launch failed: %s", hipGetErrorString(e));
  return ok();
}

// One call of the split attention (both phases or one).
specgen_status_t run_batch(const specgen_fork_batch_t* b, int32_t phase, void* out, float* out_lse, void* workspace,
                           size_t workspace_bytes, hipStream_t stream, const int32_t* ptab_sel = nullptr) {
  if (phase != SPECGEN_PHASE_ALL && phase != SPECGEN_PHASE_PARTIALS && phase != SPECGEN_PHASE_MERGE)
    return fail(SPECGEN_ERR_INVALID_ARG, "phase %d unknown", phase);
  Plan plan;
  int64_t wsf = 0;
  const specgen_status_t st = build_plan(b, &plan, &wsf, ptab_sel);
  if (st != SPECGEN_OK) return st;
  return run_plan(b, plan, wsf, phase, out, out_lse, workspace, workspace_bytes, stream);
}

// Scratch of specgen_fork_decode_attn_noalloc: the workspace of a call, in a
// device array of the library (one per GPU, held until the process ends).  In
// host code `scratch` names a host-side stand-in, not device memory: host code
// uses only the address hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) uint8_t scratch[SPECGEN_NOALLOC_SCRATCH_BYTES];
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The current device's scratch address, looked up once per device.
specgen_status_t scratch_of_current_device(void** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(SPECGEN_ERR_DEVICE, "hipGetDevice failed: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return fail(SPECGEN_ERR_UNSUPPORTED, "device %d: at most %d devices", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(SPECGEN_ERR_DEVICE, "scratch address of device %d: %s", dev, hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return ok();
}

// Multi-token prefill as a decode batch of virtual forks: query i of fork f
// becomes a fork whose suffix ends at that query's own position (S_f -
// q_len[f] + i + 1 tokens).  Where every fork of a trace has at least one
// whole block of suffix before its first query, each such fork also becomes a
// trace nested under its own trace: its prefix is those whole blocks (listed
// in the suffix table), shared by the fork's queries, and each query keeps
// only the tokens from the next block on.  The host mirrors change; the
// device arrays are shared.
struct PrefillBatch {
  specgen_fork_batch_t b;
  std::vector<int32_t> fork_off, prefix_len, prefix_table_off, parent, sel, suffix_len, suffix_table_off;
};

specgen_status_t expand_prefill(const specgen_fork_batch_t* b, const int32_t* q_len_h, PrefillBatch* x) {
  Plan plan;
  int64_t wsf = 0;
  const specgen_status_t st = build_plan(b, &plan, &wsf);   // checks the batch as given
  if (st != SPECGEN_OK) return st;
  if (!q_len_h) return fail(SPECGEN_ERR_INVALID_ARG, "q_len is NULL");
  const int T = b->num_traces, N = b->num_forks;
  int64_t nq = 0;
  for (int f = 0; f < N; ++f) {
    if (q_len_h[f] < 1 || q_len_h[f] > b->suffix_len_h[f])
      return fail(SPECGEN_ERR_INVALID_ARG, "q_len[%d] = %d must be in 1..S_f = %d", f, q_len_h[f], b->suffix_len_h[f]);
    nq += q_len_h[f];
  }
  if (nq > kMaxForks) return fail(SPECGEN_ERR_UNSUPPORTED, "%lld queries exceed %d per call", (long long)nq, kMaxForks);
  // whole suffix blocks before each fork's first query
  auto shared = [&](int f) { return (b->suffix_len_h[f] - q_len_h[f] + 1) / kBlock * kBlock; };
  // traces whose forks all get a nested trace, within the trace and depth limits
  std::vector<char> nest(T, 0);
  int budget = kMaxTraces - T;
  for (int t = 0; t < T; ++t) {
    bool ok = plan.fork_off[t + 1] - plan.fork_off[t] <= budget;
    int d = 1;
    for (int a = plan.parent[t]; a >= 0; a = plan.parent[a]) ++d;
    ok = ok && d < kMaxDepth && plan.fork_off[t + 1] > plan.fork_off[t];
    for (int f = plan.fork_off[t]; ok && f < plan.fork_off[t + 1]; ++f) ok = shared(f) >= kBlock;
    if (ok) {
      nest[t] = 1;
      budget -= plan.fork_off[t + 1] - plan.fork_off[t];
    }
  }
  x->b = *b;
  x->fork_off.assign(1, 0);
  x->prefix_len.clear();
  x->prefix_table_off.clear();
  x->parent.clear();
  x->sel.clear();
  x->suffix_len.clear();
  x->suffix_table_off.clear();
  std::vector<int32_t> pos(T, -1);   // index of each original trace in the new list
  int nv = 0;                        // virtual forks so far
  auto add_queries = [&](int f, int skip) {   // fork f's queries, each suffix starting after `skip` tokens
    for (int i = 0; i < q_len_h[f]; ++i) {
      x->suffix_len.push_back(b->suffix_len_h[f] - q_len_h[f] + i + 1 - skip);
      x->suffix_table_off.push_back(b->suffix_table_off_h[f] + skip / kBlock);
      ++nv;
    }
  };
  for (int t = 0; t < T; ++t) {
    pos[t] = (int)x->prefix_len.size();
    x->prefix_len.push_back(b->prefix_len_h[t]);
    x->prefix_table_off.push_back(b->prefix_table_off_h[t]);
    x->parent.push_back(plan.parent[t] < 0 ? -1 : pos[plan.parent[t]]);
    x->sel.push_back(0);
    if (!nest[t])
      for (int f = plan.fork_off[t]; f < plan.fork_off[t + 1]; ++f) add_queries(f, 0);
    x->fork_off.push_back(nv);
    if (nest[t]) {
      for (int f = plan.fork_off[t]; f < plan.fork_off[t + 1]; ++f) {
        x->prefix_len.push_back(shared(f));
        x->prefix_table_off.push_back(b->suffix_table_off_h[f]);
        x->parent.push_back(pos[t]);
        x->sel.push_back(1);
        add_queries(f, shared(f));
        x->fork_off.push_back(nv);
      }
    }
  }
  x->prefix_table_off.push_back(b->prefix_table_off_h[T]);
  x->suffix_table_off.push_back(b->suffix_table_off_h[N]);
  x->b.num_traces = (int32_t)x->prefix_len.size();
  x->b.num_forks = (int32_t)nq;
  x->b.fork_off_h = x->fork_off.data();
  x->b.prefix_len_h = x->prefix_len.data();
  x->b.prefix_table_off_h = x->prefix_table_off.data();
  x->b.prefix_parent_h = x->parent.data();
  x->b.suffix_len_h = x->suffix_len.data();
  x->b.suffix_table_off_h = x->suffix_table_off.data();
  return ok();
}

}  // namespace

extern "C" {

specgen_status_t specgen_fork_decode_attn_workspace_size(const specgen_fork_batch_t* b, size_t* bytes) {
  if (!bytes) return fail(SPECGEN_ERR_INVALID_ARG, "bytes is NULL");
  Plan plan;
  int64_t wsf = 0;
  const specgen_status_t st = build_plan(b, &plan, &wsf);
  if (st != SPECGEN_OK) return st;
  *bytes = (size_t)(wsf * 4);
  return ok();
}

specgen_status_t specgen_fork_decode_attn_split(const specgen_fork_batch_t* b, specgen_split_segment_t* segs,
                                                int64_t cap, int64_t* count) {
  if (!count) return fail(SPECGEN_ERR_INVALID_ARG, "count is NULL");
  if (cap < 0 || (cap > 0 && !segs)) return fail(SPECGEN_ERR_INVALID_ARG, "segs is NULL or cap < 0");
  if (!b) return fail(SPECGEN_ERR_INVALID_ARG, "batch is NULL");
  // Device arrays are not read here: stand-ins let the shared checks pass.
  specgen_fork_batch_t hb = *b;
  const void* stand_in = reinterpret_cast<const void*>(uintptr_t{256});
  if (!hb.q) hb.q = stand_in;
  if (!hb.k_pool) hb.k_pool = stand_in;
  if (!hb.v_pool) hb.v_pool = stand_in;
  if (!hb.k_scale) hb.k_scale = static_cast<const float*>(stand_in);
  if (!hb.v_scale) hb.v_scale = static_cast<const float*>(stand_in);
  for (const int32_t** a : {&hb.fork_off, &hb.prefix_len, &hb.prefix_table_off, &hb.prefix_table, &hb.suffix_len,
                            &hb.suffix_table_off, &hb.suffix_table})
    if (!*a) *a = static_cast<const int32_t*>(stand_in);
  Plan plan;
  int64_t wsf = 0;
  const specgen_status_t st = build_plan(&hb, &plan, &wsf);
  if (st != SPECGEN_OK) return st;
  int64_t n = 0;
  for (int X = 0; X < 2; ++X) {
    const PartPlan& pp = plan.part[X];
    for (int w = 0; w < pp.workers; ++w) {
      walk_range(plan, X, w, INT32_MAX, [&](const ItemRef& it, int nt, int, int, int) {
        if (n < cap) {
          specgen_split_segment_t& s = segs[n];
          const int nv = it.kind == 0 ? plan.prefix_len[it.t] : plan.suffix_len[it.f];
          s.kind = it.kind;
          s.trace = it.kind == 0 ? it.t : trace_of_fork(plan, it.f);
          s.fork = it.kind == 0 ? -1 : it.f;
          s.kv_head = it.j;
          s.row_block = it.rb;
          const int rows = it.kind == 0 ? trace_rows(plan, it.t) : plan.g;
          s.first_row = it.rb * pp.rbs;
          s.num_rows = rows - s.first_row < pp.rbs ? rows - s.first_row : pp.rbs;
          s.kernel = X;
          s.worker = w;
          s.first_token = it.tile * pp.tt;
          const int end = (it.tile + nt) * pp.tt;
          s.num_tokens = (end < nv ? end : nv) - s.first_token;
        }
        ++n;
      });
    }
  }
  *count = n;
  return ok();
}

specgen_status_t specgen_fork_decode_attn_phase(const specgen_fork_batch_t* b, int32_t phase, void* out,
                                                float* out_lse, void* workspace, size_t workspace_bytes,
                                                hipStream_t stream) {
  return run_batch(b, phase, out, out_lse, workspace, workspace_bytes, stream);
}

specgen_status_t specgen_fork_prefill_attn_workspace_size(const specgen_fork_batch_t* b, const int32_t* q_len_h,
                                                          size_t* bytes) {
  if (!bytes) return fail(SPECGEN_ERR_INVALID_ARG, "bytes is NULL");
  PrefillBatch x;
  specgen_status_t st = expand_prefill(b, q_len_h, &x);
  if (st != SPECGEN_OK) return st;
  Plan plan;
  int64_t wsf = 0;
  st = build_plan(&x.b, &plan, &wsf, x.sel.data());
  if (st != SPECGEN_OK) return st;
  *bytes = (size_t)(wsf * 4);
  return ok();
}

specgen_status_t specgen_fork_prefill_attn(const specgen_fork_batch_t* b, const int32_t* q_len_h, void* out,
                                           float* out_lse, void* workspace, size_t workspace_bytes,
                                           hipStream_t stream) {
  PrefillBatch x;
  const specgen_status_t st = expand_prefill(b, q_len_h, &x);
  if (st != SPECGEN_OK) return st;
  return run_batch(&x.b, SPECGEN_PHASE_ALL, out, out_lse, workspace, workspace_bytes, stream, x.sel.data());
}

specgen_status_t specgen_fork_decode_attn(const specgen_fork_batch_t* b, void* out, float* out_lse,
                                          void* workspace, size_t workspace_bytes, hipStream_t stream) {
  return specgen_fork_decode_attn_phase(b, SPECGEN_PHASE_ALL, out, out_lse, workspace, workspace_bytes, stream);
}

specgen_status_t specgen_fork_decode_attn_noalloc(const specgen_fork_batch_t* b, void* out, float* out_lse,
                                                  hipStream_t stream) {
  Plan plan;
  int64_t wsf = 0;
  specgen_status_t st = build_plan(b, &plan, &wsf);
  if (st != SPECGEN_OK) return st;
  if ((uint64_t)wsf * 4 > (uint64_t)SPECGEN_NOALLOC_SCRATCH_BYTES)
    return fail(SPECGEN_ERR_WORKSPACE,
                "batch needs %lld bytes of workspace, above the %llu-byte scratch of the no-allocation entry point "
                "(use specgen_fork_decode_attn with a workspace)",
                (long long)(wsf * 4), (unsigned long long)SPECGEN_NOALLOC_SCRATCH_BYTES);
  void* ws = nullptr;
  st = scratch_of_current_device(&ws);
  if (st != SPECGEN_OK) return st;
  return run_plan(b, plan, wsf, SPECGEN_PHASE_ALL, out, out_lse, ws, SPECGEN_NOALLOC_SCRATCH_BYTES, stream);
}

specgen_status_t specgen_kv_import(const specgen_kv_tensor_t* tensors, int32_t num_tensors,
                                   const int32_t* dst_block_ids, int64_t n, int64_t num_dst_blocks,
                                   int32_t* bad_id_count, hipStream_t stream) {
  if (!tensors) return fail(SPECGEN_ERR_INVALID_ARG, "tensors is NULL");
  if (num_tensors < 1 || num_tensors > 4) return fail(SPECGEN_ERR_INVALID_ARG, "num_tensors %d not in 1..4", num_tensors);
  if (n < 0 || n > INT32_MAX) return fail(SPECGEN_ERR_INVALID_ARG, "n %lld out of range", (long long)n);
  if (num_dst_blocks < 0) return fail(SPECGEN_ERR_INVALID_ARG, "num_dst_blocks must be >= 0");
  if (n > 0 && !dst_block_ids) return fail(SPECGEN_ERR_INVALID_ARG, "dst_block_ids is NULL");
  BlockCopyArgs a;
  std::memset(&a, 0, sizeof a);
  for (int i = 0; i < num_tensors; ++i) {
    const specgen_kv_tensor_t& t = tensors[i];
    if (t.block_bytes <= 0 || (t.block_bytes & 3))
      return fail(SPECGEN_ERR_INVALID_ARG, "tensor %d: block_bytes %lld must be > 0 and a multiple of 4", i,
                  (long long)t.block_bytes);
    if (n > 0 && (!t.dst_pool || !t.src_staging)) return fail(SPECGEN_ERR_INVALID_ARG, "tensor %d: NULL pointer", i);
    const uintptr_t al = (t.block_bytes & 15) ? 3 : 15;
    if (((uintptr_t)t.dst_pool & al) || ((uintptr_t)t.src_staging & al))
      return fail(SPECGEN_ERR_INVALID_ARG, "tensor %d: pointers must be aligned to the copy vector", i);
    a.t[i].pool = static_cast<uint8_t*>(t.dst_pool);
    a.t[i].staging = const_cast<uint8_t*>(static_cast<const uint8_t*>(t.src_staging));
    a.t[i].block_bytes = t.block_bytes;
  }
  a.num_tensors = num_tensors;
  a.ids = dst_block_ids;
  a.n = n;
  a.num_pool_blocks = num_dst_blocks;
  a.bad_id_count = bad_id_count;
  const hipError_t e = launch_kv_import(a, stream);
  if (e != hipSuccess) return fail(SPECGEN_ERR_DEVICE, "kernel launch failed: %s", hipGetErrorString(e));
  return ok();
}

specgen_status_t specgen_kv_export(const specgen_kv_export_tensor_t* tensors, int32_t num_tensors,
                                   const int32_t* src_block_ids, int64_t n, int64_t num_src_blocks,
                                   int32_t* bad_id_count, hipStream_t stream) {
  if (!tensors) return fail(SPECGEN_ERR_INVALID_ARG, "tensors is NULL");
  if (num_tensors < 1 || num_tensors > 4) return fail(SPECGEN_ERR_INVALID_ARG, "num_tensors %d not in 1..4", num_tensors);
  if (n < 0 || n > INT32_MAX) return fail(SPECGEN_ERR_INVALID_ARG, "n %lld out of range", (long long)n);
  if (num_src_blocks < 0) return fail(SPECGEN_ERR_INVALID_ARG, "num_src_blocks must be >= 0");
  if (n > 0 && !src_block_ids) return fail(SPECGEN_ERR_INVALID_ARG, "src_block_ids is NULL");
  BlockCopyArgs a;
  std::memset(&a, 0, sizeof a);
  for (int i = 0; i < num_tensors; ++i) {
    const specgen_kv_export_tensor_t& t = tensors[i];
    if (t.block_bytes <= 0 || (t.block_bytes & 3))
      return fail(SPECGEN_ERR_INVALID_ARG, "tensor %d: block_bytes %lld must be > 0 and a multiple of 4", i,
                  (long long)t.block_bytes);
    if (n > 0 && (!t.dst_staging || !t.src_pool)) return fail(SPECGEN_ERR_INVALID_ARG, "tensor %d: NULL pointer", i);
    const uintptr_t al = (t.block_bytes & 15) ? 3 : 15;
    if (((uintptr_t)t.dst_staging & al) || ((uintptr_t)t.src_pool & al))
      return fail(SPECGEN_ERR_INVALID_ARG, "tensor %d: pointers must be aligned to the copy vector", i);
    a.t[i].pool = const_cast<uint8_t*>(static_cast<const uint8_t*>(t.src_pool));
    a.t[i].staging = static_cast<uint8_t*>(t.dst_staging);
    a.t[i].block_bytes = t.block_bytes;
  }
  a.num_tensors = num_tensors;
  a.ids = src_block_ids;
  a.n = n;
  a.num_pool_blocks = num_src_blocks;
  a.bad_id_count = bad_id_count;
  const hipError_t e = launch_kv_export(a, stream);
  if (e != hipSuccess) return fail(SPECGEN_ERR_DEVICE, "kernel launch failed: %s", hipGetErrorString(e));
  return ok();
}

specgen_status_t specgen_kv_append(const specgen_kv_append_t* p, hipStream_t stream) {
  if (!p) return fail(SPECGEN_ERR_INVALID_ARG, "append descriptor is NULL");
  if (p->num_forks < 0) return fail(SPECGEN_ERR_INVALID_ARG, "num_forks must be >= 0 (got %d)", p->num_forks);
  if (p->num_kv_heads < 1) return fail(SPECGEN_ERR_INVALID_ARG, "num_kv_heads must be >= 1");
  if (p->head_dim < 1 || p->head_dim > 1024)
    return fail(SPECGEN_ERR_INVALID_ARG, "head_dim %d not in 1..1024", p->head_dim);
  if (p->kv_dtype != SPECGEN_BF16 && p->kv_dtype != SPECGEN_FP8_E4M3)
    return fail(SPECGEN_ERR_UNSUPPORTED, "kv_dtype %d not supported", p->kv_dtype);
  if (p->num_blocks < 1) return fail(SPECGEN_ERR_INVALID_ARG, "num_blocks must be >= 1");
  if ((int64_t)p->num_forks * p->num_kv_heads > 4LL * INT32_MAX)
    return fail(SPECGEN_ERR_INVALID_ARG, "num_forks * num_kv_heads too large");
  const int es = p->kv_dtype == SPECGEN_BF16 ? 2 : 1;
  if (p->num_forks > 0) {
    if (!p->k_pool || !p->v_pool || !p->k_new || !p->v_new || !p->pos || !p->suffix_table_off || !p->suffix_table)
      return fail(SPECGEN_ERR_INVALID_ARG, "NULL pointer in append descriptor");
    if (es == 2 && (((uintptr_t)p->k_pool | (uintptr_t)p->v_pool | (uintptr_t)p->k_new | (uintptr_t)p->v_new) & 1))
      return fail(SPECGEN_ERR_INVALID_ARG, "bf16 arrays must be 2-byte aligned");
  }
  AppendArgs a;
  a.k_pool = static_cast<uint8_t*>(p->k_pool);
  a.v_pool = static_cast<uint8_t*>(p->v_pool);
  a.k_new = static_cast<const uint8_t*>(p->k_new);
  a.v_new = static_cast<const uint8_t*>(p->v_new);
  a.pos = p->pos;
  a.suffix_table_off = p->suffix_table_off;
  a.suffix_table = p->suffix_table;
  a.bad_count = p->bad_count;
  a.num_blocks = p->num_blocks;
  a.num_forks = p->num_forks;
  a.num_kv_heads = p->num_kv_heads;
  a.head_dim = p->head_dim;
  a.elem_bytes = es;
  const hipError_t e = launch_kv_append(a, stream);
  if (e != hipSuccess) return fail(SPECGEN_ERR_DEVICE, "kernel launch failed: %s", hipGetErrorString(e));
  return ok();
}

specgen_status_t specgen_lse_merge(const float* o_parts, const float* lse_parts, int32_t num_parts, int64_t rows,
                                   int32_t head_dim, void* out, int32_t out_dtype, float* out_lse,
                                   hipStream_t stream) {
  if (num_parts < 1) return fail(SPECGEN_ERR_INVALID_ARG, "num_parts must be >= 1");
  if (rows < 0) return fail(SPECGEN_ERR_INVALID_ARG, "rows must be >= 0");
  if (head_dim < 1 || head_dim > 1024) return fail(SPECGEN_ERR_INVALID_ARG, "head_dim %d not in 1..1024", head_dim);
  if (out_dtype != SPECGEN_BF16 && out_dtype != SPECGEN_FP32)
    return fail(SPECGEN_ERR_INVALID_ARG, "out_dtype must be BF16 or FP32");
  if (rows > 0 && (!o_parts || !lse_parts || !out)) return fail(SPECGEN_ERR_INVALID_ARG, "NULL pointer");
  if (rows > (int64_t)UINT32_MAX * 4) return fail(SPECGEN_ERR_UNSUPPORTED, "too many rows");
  const hipError_t e = launch_lse_merge(o_parts, lse_parts, num_parts, rows, head_dim, out,
                                        out_dtype == SPECGEN_BF16, out_lse, stream);
  if (e != hipSuccess) return fail(SPECGEN_ERR_DEVICE, "kernel launch failed: %s", hipGetErrorString(e));
  return ok();
}

const char* specgen_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
