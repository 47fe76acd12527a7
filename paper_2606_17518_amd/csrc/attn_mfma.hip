// attn_mfma.hip -- the shared-prefix (and suffix) partial-attention kernel on
// gfx950 bf16 matrix cores.
//
// One workgroup = one worker of the MFMA partition (plan.h): it walks a
// contiguous range of tiles, each tile being TT consecutive tokens of one work
// item.  For a prefix item the rows are every (fork, q head) pair of a GQA
// group of one trace, so the tile's K/V is read from HBM once and used by all
// forks -- the shared reasoning prefix is read once per step instead of once
// per fork (forks reuse the prefix cache, Sec. 4.2 / Sec. 8.7).  For a suffix
// item the rows are one fork's g query heads (padded to 32 rows per wave).
//
// This kernel serves E4M3 KV (bf16 KV has its own kernel, attn_bf16.hip).
// Data path per tile (D=128: 64 tokens, 8 KiB of K codes + 8 KiB of V codes):
//   HBM --global_load_dwordx2--> VGPRs (three tiles in flight) --exact E4M3 to
//   bf16, ds_write_b128--> swizzled LDS --ds_read_b128 (K rows; V^T rows, as V
//   is stored transposed)--> MFMA.
// Per 32-token slab and 16-row N-tile, S^T = K Q^T on v_mfma_f32_16x16x32_bf16
// (A = 16 keys x 32 dims, B = Q^T 32 dims x 16 rows); the keys of the two S^T
// tiles are taken in the order that makes each lane's scores the 8
// consecutive tokens PV consumes, so the scores feed O^T = V^T P^T (A = V^T 16
// dims x 32 tokens, one 16-byte LDS read per lane, B = P^T) without a shuffle.
// Online softmax in fp32 per row; each worker writes one normalised partial
// (o, lse) per item it touched, merged later by the log-sum-exp rule.
#include "kernels.h"
#include "worker.h"

namespace specgen {

// The running max moves only when a new score would give a probability above
// 2^kRescaleLog2 relative to it.
constexpr float kRescaleLog2 = 8.f;

template <int D, bool FP8>
struct MfmaCfg {
  static constexpr int kThreads = 256;
  static constexpr int kWaves = 4;
  static constexpr int kTT = (D == 128) ? 64 : 128;   // tokens per tile
  static constexpr int kRowB = D * 2;                 // LDS bytes per token row (bf16)
  static constexpr int kCPR = kRowB / 16;             // 16-byte chunks per LDS row
  static constexpr int kTileB = kTT * kRowB;          // LDS bytes of one K or V tile
  static constexpr int kSliceB = 16 * kRowB;          // LDS bytes of one block's V^T slice
  static constexpr int kLoads = kTileB / 16 / kThreads;  // chunks per thread per tensor
  static constexpr int kGElem = FP8 ? 1 : 2;          // pool bytes per element
  static constexpr int kGChunk = 8 * kGElem;          // pool bytes per LDS chunk
  static constexpr int kIdsPerTile = kTT / 16;
  static constexpr int kStageB = 2 * kTileB;
  static constexpr int kItemCap = 64;
  static constexpr int kIdCap = 2048;
  static constexpr int kTileCap = kIdCap / kIdsPerTile;
  // LDS layout
  static constexpr int kOffStage0 = 0;
  static constexpr int kOffStage1 = kStageB;
  static constexpr int kOffComb = 2 * kStageB;                 // [2 rg][32 rows][D] f32
  static constexpr int kOffCombML = kOffComb + 2 * 32 * D * 4; // [2 rg][32] m, then l
  static constexpr int kOffItems = kOffCombML + 2 * 2 * 32 * 4;
  static constexpr int kOffIds = kOffItems + kItemCap * kItemInts * 4;
  static constexpr int kOffScales = kOffIds + kIdCap * 4;      // E4M3: k then v scale per id
  static constexpr int kLdsBytes = kOffScales + (FP8 ? 2 * kIdCap * 4 : 0);
  static_assert(kLoads * 16 * kThreads == kTileB, "tile must split evenly over threads");
  static_assert(kLdsBytes <= 163840, "LDS budget");
};

template <int D, bool FP8>
__global__ void __launch_bounds__(256, 1) attn_mfma_kernel(const AttnArgs a, const Plan plan_arg) {
  using C = MfmaCfg<D, FP8>;
  constexpr int TT = C::kTT;
  constexpr int KS = D / 32;   // k-steps of S^T
  constexpr int DT = D / 16;   // d-tiles of O^T
  __shared__ __attribute__((aligned(16))) uint8_t lds[C::kLdsBytes];
  __shared__ Plan splan;
  plan_to_lds<256>(plan_arg, splan);
  const Plan& plan = splan;
  int32_t* items = reinterpret_cast<int32_t*>(lds + C::kOffItems);
  int32_t* ids = reinterpret_cast<int32_t*>(lds + C::kOffIds);

  const PartPlan& pp = plan.part[kPartMfma];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int w = blockIdx.x;
  float* scales = FP8 ? reinterpret_cast<float*>(lds + C::kOffScales) : nullptr;
  const WorkerRange wr = worker_prepass<C::kThreads, C::kItemCap, C::kIdsPerTile, C::kTileCap>(
      a, plan, kPartMfma, w, items, ids, scales);
  const int R = wr.R;
  const int nitems = wr.nitems;
  const int first_ord = wr.first_ord;
  if (R <= 0) return;

  // ---- loads: tile r of the range into registers ------------------------------
  // Inside a pool block, kv head j's K is 16 token rows of D values and its V
  // is D rows of 16 token values (V transposed).  A K chunk is 8 values of one
  // token; a V chunk is 8 tokens of one dim (half h of row d of a block slice).
  typedef typename std::conditional<FP8, u32x2, u32x4>::type chunk_t;
  const int64_t slice_b = (int64_t)16 * D * C::kGElem;   // one block's slice of one kv head
  auto tile_item = [&](int r) { return item_of_tile(items, nitems, r); };
  // Loads are issued unconditionally so the compiler can count outstanding
  // vector loads exactly across the pipeline; past the range end every lane
  // re-reads the first 16 bytes of q (one cached line, no HBM traffic).
  auto issue = [&](chunk_t (&rk)[C::kLoads], chunk_t (&rv)[C::kLoads], int r) {
    const bool real = r < R;
    const int rr = real ? r : R - 1;
    const int ii = uniform(tile_item(rr));
    const int32_t* d = items + ii * kItemInts;
    const int j = uniform(d[IT_J]);
    const int nv = uniform(d[IT_NVALID]);
    const int tbase = (uniform(d[IT_TILE0]) + (rr - uniform(d[IT_RTILE0]))) * TT;
    const uint8_t* kp = real ? a.k_pool : reinterpret_cast<const uint8_t*>(a.q);
    const uint8_t* vp = real ? a.v_pool : reinterpret_cast<const uint8_t*>(a.q);
#pragma unroll
    for (int it = 0; it < C::kLoads; ++it) {
      const int c = it * C::kThreads + tid;
      // K: token row tok, chunk part
      const int tok = c / C::kCPR;
      const int part = c % C::kCPR;
      int ti = tbase + tok;
      if (ti >= nv) ti = nv - 1;   // rows past the item's end re-read its last valid token
      const int kblk = ids[rr * C::kIdsPerTile + tok / 16];
      int64_t koff = ((int64_t)kblk * plan.Hkv + j) * slice_b + (int64_t)(ti & 15) * D * C::kGElem + part * C::kGChunk;
      // V: block kb of the tile, row d, half h
      const int kb = c / (2 * D);
      const int dd = (c % (2 * D)) >> 1;
      const int h = c & 1;
      const int vblk = ids[rr * C::kIdsPerTile + kb];
      int64_t voff = ((int64_t)vblk * plan.Hkv + j) * slice_b + (int64_t)(dd * 16 + 8 * h) * C::kGElem;
      koff = real ? koff : 0;
      voff = real ? voff : 0;
      rk[it] = *reinterpret_cast<const chunk_t*>(kp + koff);
      rv[it] = *reinterpret_cast<const chunk_t*>(vp + voff);
    }
  };
  auto to_lds_chunk = [&](const chunk_t& v) -> u32x4 {
    if constexpr (FP8) {
      // exact E4M3 -> bf16: the hardware fp8 -> f32 conversion, then the upper half
      u32x4 o;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const uint32_t wv = v[h];
        f32x2 lo = __builtin_amdgcn_cvt_pk_f32_fp8(wv, false);
        f32x2 hi = __builtin_amdgcn_cvt_pk_f32_fp8(wv, true);
        o[2 * h] = (__float_as_uint(lo[0]) >> 16) | (__float_as_uint(lo[1]) & 0xFFFF0000u);
        o[2 * h + 1] = (__float_as_uint(hi[0]) >> 16) | (__float_as_uint(hi[1]) & 0xFFFF0000u);
      }
      return o;
    } else {
      return v;
    }
  };
  // V chunk c of tile r lands at LDS position 2d + (h ^ bit 3 of d) of its block
  // slice (a 16-lane read of 16 consecutive dims hits distinct banks); values of
  // tokens past the item's end may be any bits and are zeroed here.
  auto store = [&](const chunk_t (&rk)[C::kLoads], const chunk_t (&rv)[C::kLoads], int stage_off, int r) {
    const int rr = r < R ? r : R - 1;
    const int32_t* d = items + uniform(tile_item(rr)) * kItemInts;
    const int nv = uniform(d[IT_NVALID]);
    const int tbase = (uniform(d[IT_TILE0]) + (rr - uniform(d[IT_RTILE0]))) * TT;
#pragma unroll
    for (int it = 0; it < C::kLoads; ++it) {
      const int c = it * C::kThreads + tid;
      const int tok = c / C::kCPR;
      const int part = c % C::kCPR;
      const int kpos = tok * C::kRowB + ((part ^ swz_k<C::kCPR>(tok)) << 4);
      const int kb = c / (2 * D);
      const int dd = (c % (2 * D)) >> 1;
      const int h = c & 1;
      const int vpos = kb * C::kSliceB + 16 * (2 * dd + (h ^ ((dd >> 3) & 1)));
      u32x4 vv = to_lds_chunk(rv[it]);
      const int t0 = tbase + kb * 16 + 8 * h;   // first token of the chunk
#pragma unroll
      for (int e2 = 0; e2 < 4; ++e2)
        vv[e2] &= (t0 + 2 * e2 < nv ? 0x0000FFFFu : 0u) | (t0 + 2 * e2 + 1 < nv ? 0xFFFF0000u : 0u);
      *reinterpret_cast<SG_LDS u32x4*>((SG_LDS uint8_t*)lds + stage_off + kpos) = to_lds_chunk(rk[it]);
      *reinterpret_cast<SG_LDS u32x4*>((SG_LDS uint8_t*)lds + stage_off + C::kTileB + vpos) = vv;
    }
  };

  // ---- per-wave compute state -----------------------------------------------------
  const int G = lane >> 4;     // 16-lane group
  const int ln = lane & 15;    // row within an N-tile / key within an S^T tile
  // Lane-constant parts of the LDS addresses (slab bases are multiples of 32):
  // the key this lane feeds to S^T tile a (tile b is 4 keys later) and its
  // swizzle, and this lane's V^T operand position: block sb/16 + G/2 of the
  // tile, row d = 16 dt + ln, half G & 1.
  const int k_lane_tok = 8 * (ln >> 2) + (ln & 3);
  const int k_lane_swz = swz_k<C::kCPR>(k_lane_tok);
  const int v_lane_off = (G >> 1) * C::kSliceB + 32 * ln + 16 * ((G & 1) ^ ((ln >> 3) & 1));
  bf16x8 qop[2][KS];
  f32x4 acc[2][DT];
  float m_run[2], l_run[2];
  int rg = 0, tg = 0, ntg = 1, active = 0, nrows = 0;
  float ks_scale = 1.f;        // E4M3: K block scale folded into the scores
  (void)ks_scale;

  auto begin_item = [&](const int32_t* d) {
    nrows = uniform(d[IT_NROWS]);
    if (nrows > 64) { ntg = 1; rg = wave; tg = 0; }
    else { ntg = 2; rg = wave & 1; tg = wave >> 1; }
    active = rg * 32 < nrows;
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
      const int rr = rg * 32 + nt * 16 + ln;
      int fork = 0, h = 0;
      item_row(plan, d, rr, &fork, &h);
      const bool ok = active && rr < nrows;
      // unconditional loads (padded rows read row 0 and are zeroed) keep the
      // number of outstanding loads the same on every path
      const uint16_t* qrow = a.q + (ok ? ((int64_t)fork * plan.Hq + h) * D : 0);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        u32x4 v = *reinterpret_cast<const u32x4*>(qrow + ks * 32 + G * 8);
        if (!ok) v = u32x4{0u, 0u, 0u, 0u};
        qop[nt][ks] = __builtin_bit_cast(bf16x8, v);
      }
      m_run[nt] = -INFINITY;
      l_run[nt] = 0.f;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) acc[nt][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    wait_vmem();
  };

  auto compute_tile = [&](int stage_off, const int32_t* d, int r) {
    if (!active) return;
    const int tile_in_item = uniform(d[IT_TILE0]) + (r - uniform(d[IT_RTILE0]));
    const int nv = uniform(d[IT_NVALID]);
    const int valid = (nv - tile_in_item * TT) < TT ? (nv - tile_in_item * TT) : TT;
    const int ntok = TT / ntg;
    const int tok0 = tg * ntok;
    const SG_LDS uint8_t* kb = (const SG_LDS uint8_t*)lds + stage_off;
    const SG_LDS uint8_t* vb = kb + C::kTileB;
    for (int sb = tok0; sb < tok0 + ntok; sb += 32) {
      if (sb >= valid) break;
      f32x4 s[2][2];
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) s[u][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
      // slab bases are multiples of 32, so the swizzles depend on the lane only
      const SG_LDS uint8_t* ka_row = kb + (sb + k_lane_tok) * C::kRowB;
      const SG_LDS uint8_t* kb_row = ka_row + 4 * C::kRowB;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const int cho = (((4 * ks + G) ^ k_lane_swz) << 4);
        const u32x4 ka = *reinterpret_cast<const SG_LDS u32x4*>(ka_row + cho);
        const u32x4 kbv = *reinterpret_cast<const SG_LDS u32x4*>(kb_row + cho);
        const bf16x8 A0 = __builtin_bit_cast(bf16x8, ka);
        const bf16x8 A1 = __builtin_bit_cast(bf16x8, kbv);
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) {
          s[0][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A0, qop[nt][ks], s[0][nt], 0, 0, 0);
          s[1][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A1, qop[nt][ks], s[1][nt], 0, 0, 0);
        }
      }
      // lane (G, ln) now holds, for row ln of each N-tile, the scores of keys sb+8G+0..7
      if constexpr (FP8) {
        const float ksc = scales[r * C::kIdsPerTile + (sb + 8 * G) / 16];
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
          for (int nt = 0; nt < 2; ++nt) s[u][nt] *= ksc;
      }
      if (sb + 32 > valid) {
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (sb + 8 * G + 4 * u + e >= valid) {
              s[u][0][e] = -INFINITY;
              s[u][1][e] = -INFINITY;
            }
      }
      bf16x8 pop[2];
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) {
        float mx = fmaxf(fmaxf(fmaxf(s[0][nt][0], s[0][nt][1]), fmaxf(s[0][nt][2], s[0][nt][3])),
                         fmaxf(fmaxf(s[1][nt][0], s[1][nt][1]), fmaxf(s[1][nt][2], s[1][nt][3])));
        mx = rows4_max(mx);
        // Lazy rescaling: the reference max only moves when a score exceeds it
        // by more than 2^kRescaleLog2 in probability, so P <= 2^8 stays exact
        // enough in bf16 and fp32 and the accumulator is rarely touched.
        if (__builtin_amdgcn_ballot_w64(mx * a.c_log2 > m_run[nt] * a.c_log2 + kRescaleLog2)) {
          const float m_new = fmaxf(m_run[nt], mx);
          const float alpha = __builtin_amdgcn_exp2f((m_run[nt] - m_new) * a.c_log2);
          m_run[nt] = m_new;
          l_run[nt] *= alpha;
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) scale_acc(acc[nt][dt], alpha);
        }
        const float mc = m_run[nt] * a.c_log2;
        float p[8];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          p[e] = __builtin_amdgcn_exp2f(fmaf(s[0][nt][e], a.c_log2, -mc));
          p[4 + e] = __builtin_amdgcn_exp2f(fmaf(s[1][nt][e], a.c_log2, -mc));
        }
        l_run[nt] += ((p[0] + p[1]) + (p[2] + p[3])) + ((p[4] + p[5]) + (p[6] + p[7]));
        if constexpr (FP8) {
          const float vsc = scales[C::kIdCap + r * C::kIdsPerTile + (sb + 8 * G) / 16];
#pragma unroll
          for (int e = 0; e < 8; ++e) p[e] *= vsc;
        }
        u32x4 pk;
        pk[0] = pack_bf16x2(p[0], p[1]);
        pk[1] = pack_bf16x2(p[2], p[3]);
        pk[2] = pack_bf16x2(p[4], p[5]);
        pk[3] = pack_bf16x2(p[6], p[7]);
        pop[nt] = __builtin_bit_cast(bf16x8, pk);
      }
      // O^T += V^T P^T: lane (G, ln) reads V[sb+8G+0..7][16dt+ln] in one 16-byte load
      const SG_LDS uint8_t* vrow = vb + (sb >> 4) * C::kSliceB + v_lane_off;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const bf16x8 A = *reinterpret_cast<const SG_LDS bf16x8*>(vrow + dt * 512);
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) acc[nt][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, pop[nt], acc[nt][dt], 0, 0, 0);
      }
    }
  };

  float* comb = reinterpret_cast<float*>(lds + C::kOffComb);
  float* comb_m = reinterpret_cast<float*>(lds + C::kOffCombML);
  float* comb_l = comb_m + 2 * 32;
  auto finish_item = [&](const int32_t* d) {
    float lrow[2];
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) lrow[nt] = rows4_sum(l_run[nt]);
    if (ntg == 2) {
      if (tg == 1 && active) {
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) {
          const int row = nt * 16 + ln;
#pragma unroll
          for (int dt = 0; dt < DT; ++dt)
            *reinterpret_cast<f32x4*>(comb + (rg * 32 + row) * D + dt * 16 + 4 * G) = acc[nt][dt];
          if (G == 0) {
            comb_m[rg * 32 + row] = m_run[nt];
            comb_l[rg * 32 + row] = lrow[nt];
          }
        }
      }
      lds_barrier();
      if (tg == 0 && active) {
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) {
          const int row = nt * 16 + ln;
          const float m1 = comb_m[rg * 32 + row];
          const float l1 = comb_l[rg * 32 + row];
          const float m = fmaxf(m_run[nt], m1);
          const float mc = (m == -INFINITY) ? 0.f : m * a.c_log2;
          const float a0 = __builtin_amdgcn_exp2f(m_run[nt] * a.c_log2 - mc);
          const float a1 = __builtin_amdgcn_exp2f(m1 * a.c_log2 - mc);
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) {
            const f32x4 o1 = *reinterpret_cast<const f32x4*>(comb + (rg * 32 + row) * D + dt * 16 + 4 * G);
            acc[nt][dt] = acc[nt][dt] * a0 + o1 * a1;
          }
          lrow[nt] = lrow[nt] * a0 + l1 * a1;
          m_run[nt] = m;
        }
      }
      lds_barrier();
    }
    if (tg == 0 && active) {
      const int k = uniform(d[IT_ORD]) - first_ord;
      const int64_t slot = slot_of(pp, w, k);
      if (slot >= 0) {
        float* o = a.ws + pp.o_base + slot * pp.slot_rows * D;
        float* ls = a.ws + pp.lse_base + slot * pp.slot_rows;
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) {
          const int rr = rg * 32 + nt * 16 + ln;
          if (rr < nrows) {
            const float inv = 1.f / lrow[nt];
#pragma unroll
            for (int dt = 0; dt < DT; ++dt)
              *reinterpret_cast<f32x4*>(o + rr * D + dt * 16 + 4 * G) = acc[nt][dt] * inv;
            if (G == 0) ls[rr] = m_run[nt] * a.sm_scale + __logf(lrow[nt]);
          }
        }
      }
    }
  };

  // ---- pipeline: tile t is staged through LDS stage t % 2 and register set
  // t % 3, so three tiles are in flight while one is computed
  chunk_t kA[C::kLoads], vA[C::kLoads], kB[C::kLoads], vB[C::kLoads], kC[C::kLoads], vC[C::kLoads];
  auto stage_of = [&](int t) { return (t & 1) ? C::kOffStage1 : C::kOffStage0; };
  issue(kA, vA, 0);
  issue(kB, vB, 1);
  issue(kC, vC, 2);
  store(kA, vA, stage_of(0), 0);
  issue(kA, vA, 3);
  lds_barrier();

  int cur = -1;   // item index being accumulated
  auto step = [&](int r, int stage_off) {
    if (r >= R) return;
    const int ii = uniform(tile_item(r));
    const int32_t* d = items + ii * kItemInts;
    if (ii != cur) {
      begin_item(d);
      cur = ii;
    }
    compute_tile(stage_off, d, r);
    if (r - uniform(d[IT_RTILE0]) == uniform(d[IT_NTILE]) - 1) finish_item(d);
  };
  // Stores are unconditional too: a stage written past the range end is never read.
  // Single-exit loop over tile triples; step() ignores tiles past the range and
  // the loads behind them are harmless re-reads of q.
  for (int r = 0; r < R; r += 3) {
    step(r, stage_of(r));
    store(kB, vB, stage_of(r + 1), r + 1);
    issue(kB, vB, r + 4);
    lds_barrier();
    step(r + 1, stage_of(r + 1));
    store(kC, vC, stage_of(r + 2), r + 2);
    issue(kC, vC, r + 5);
    lds_barrier();
    step(r + 2, stage_of(r + 2));
    store(kA, vA, stage_of(r + 3), r + 3);
    issue(kA, vA, r + 6);
    lds_barrier();
  }
}

template <int D, bool FP8>
hipError_t launch_attn_mfma_t(const AttnArgs& a, const Plan& plan, hipStream_t stream) {
  const int W = plan.part[kPartMfma].workers;
  if (W <= 0) return hipSuccess;
  hipLaunchKernelGGL((attn_mfma_kernel<D, FP8>), dim3(W), dim3(256), 0, stream, a, plan);
  return hipGetLastError();
}

int mfma_tile_tokens(int D, bool fp8) {
  (void)fp8;
  return D == 128 ? MfmaCfg<128, false>::kTT : MfmaCfg<64, false>::kTT;
}
int mfma_item_cap() { return MfmaCfg<128, false>::kItemCap; }
// bf16 KV runs on the four-wave 64-rows-per-wave kernel (attn_bf16.hip).
int mfma_tile_cap(int D, bool fp8) {
  if (!fp8) return bf16_tile_cap(D);
  return D == 128 ? MfmaCfg<128, true>::kTileCap : MfmaCfg<64, true>::kTileCap;
}

hipError_t launch_attn_mfma_any(const AttnArgs& a, const Plan& plan, bool fp8, hipStream_t stream) {
  if (!fp8) return launch_attn_bf16(a, plan, stream);
  return plan.D == 128 ? launch_attn_mfma_t<128, true>(a, plan, stream) : launch_attn_mfma_t<64, true>(a, plan, stream);
}

}  // namespace specgen
