// attn_dot.hip -- the wavefront dot-product partial-attention kernel, for
// work items with fewer rows than a 16-row matrix-core tile (a prefix shared
// by too few forks x heads, or any item when the dot path is forced).
//
// Same work split and pre-pass as the MFMA kernel (worker.h).  A tile is 64
// tokens; each wave takes 16 of them as four independent streams of 4 tokens
// (16 lanes per token, D/16 dims per lane).  Scores use v_dot2_f32_bf16 on
// packed bf16 pairs and a 16-lane butterfly sum; each stream keeps its own
// online-softmax state (m, l, o) per row.  Streams are combined with
// cross-lane shuffles, waves through LDS, and one normalised partial (o, lse)
// per item is written for the log-sum-exp merge.  K/V come straight from HBM
// into registers, one tile ahead of the math (V, stored transposed, as the
// stream's 4 consecutive tokens of each of the lane's dims).
#include "worker.h"

namespace specgen {

template <int D, bool FP8>
struct DotCfg {
  static constexpr int kThreads = 256;
  static constexpr int kTT = 64;                 // tokens per tile
  static constexpr int kRows = 16;               // max rows per item
  static constexpr int kDPL = D / 16;            // dims per lane (8 or 4)
  static constexpr int kTB = 4;                  // tokens per stream per tile
  static constexpr int kGElem = FP8 ? 1 : 2;
  static constexpr int kIdsPerTile = kTT / 16;
  static constexpr int kItemCap = 64;
  static constexpr int kIdCap = 2048;
  static constexpr int kTileCap = kIdCap / kIdsPerTile;
  static constexpr int kOffComb = 0;                           // [4 waves][16 rows][D] f32
  static constexpr int kOffML = kOffComb + 4 * kRows * D * 4;   // [4 waves][16] m, then l
  static constexpr int kOffItems = kOffML + 2 * 4 * kRows * 4;
  static constexpr int kOffIds = kOffItems + kItemCap * kItemInts * 4;
  static constexpr int kOffScales = kOffIds + kIdCap * 4;      // E4M3: k then v scale per id
  static constexpr int kLdsBytes = kOffScales + (FP8 ? 2 * kIdCap * 4 : 0);
};

// kDPL pool elements of one token as packed bf16 pairs (E4M3 decoded exactly).
template <int DPL, bool FP8>
struct TokVec {
  uint32_t w[DPL / 2];
};

template <int D, bool FP8>
__global__ void __launch_bounds__(256, 1) attn_dot_kernel(const AttnArgs a, const Plan plan_arg) {
  using C = DotCfg<D, FP8>;
  constexpr int DPL = C::kDPL;
  constexpr int NP = DPL / 2;     // bf16 pairs per lane
  constexpr int RWS = C::kRows;
  constexpr int TB = C::kTB;
  __shared__ __attribute__((aligned(16))) uint8_t lds[C::kLdsBytes];
  __shared__ Plan splan;
  plan_to_lds<256>(plan_arg, splan);
  const Plan& plan = splan;
  int32_t* items = reinterpret_cast<int32_t*>(lds + C::kOffItems);
  int32_t* ids = reinterpret_cast<int32_t*>(lds + C::kOffIds);
  const PartPlan& pp = plan.part[kPartDot];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int grp = lane >> 4;      // token stream within the wave
  const int sub = lane & 15;      // dims [sub*DPL, +DPL)
  const int w = blockIdx.x;
  float* scales = FP8 ? reinterpret_cast<float*>(lds + C::kOffScales) : nullptr;
  const WorkerRange wr = worker_prepass<C::kThreads, C::kItemCap, C::kIdsPerTile, C::kTileCap>(
      a, plan, kPartDot, w, items, ids, scales);
  const int R = wr.R;
  if (R <= 0) return;
  const int nitems = wr.nitems;

  // Inside a pool block, kv head j's K is 16 token rows of D values and its V
  // is D rows of 16 token values (V transposed).  A lane loads, for each of
  // its stream's TB tokens, its DPL dims of K, and for each of its DPL dims the
  // stream's TB consecutive tokens of V.
  const int64_t slice_b = (int64_t)16 * D * C::kGElem;
  constexpr int VW = TB * C::kGElem / 4;   // 32-bit words of TB tokens of one V dim
  typedef typename std::conditional<FP8, uint32_t[DPL / 4], uint32_t[DPL / 2]>::type raw_t;
  struct Raw {
    raw_t k[TB];
    uint32_t v[DPL][VW];
  };
  // this lane's tokens of tile r: wave*16 + grp*4 + i (one 16-token block per wave)
  auto load_tile = [&](Raw& raw, int r) {
    if (r >= R) return;
    const int ii = uniform(item_of_tile(items, nitems, r));
    const int32_t* d = items + ii * kItemInts;
    const int j = uniform(d[IT_J]);
    const int nv = uniform(d[IT_NVALID]);
    const int tbase = (uniform(d[IT_TILE0]) + (r - uniform(d[IT_RTILE0]))) * C::kTT;
    // clamped tokens sit in the item's last block, which ids[] already holds
    const int blk = ids[r * C::kIdsPerTile + wave];
    const uint8_t* kslice = a.k_pool + ((int64_t)blk * plan.Hkv + j) * slice_b;
    const uint8_t* vslice = a.v_pool + ((int64_t)blk * plan.Hkv + j) * slice_b;
#pragma unroll
    for (int i = 0; i < TB; ++i) {
      int ti = tbase + wave * 16 + grp * TB + i;
      if (ti >= nv) ti = nv - 1;
      const int64_t off = (int64_t)(ti & 15) * D * C::kGElem + sub * DPL * C::kGElem;
      if constexpr (FP8) {
        if constexpr (DPL == 8) {
          const u32x2 kk = *reinterpret_cast<const u32x2*>(kslice + off);
          raw.k[i][0] = kk[0]; raw.k[i][1] = kk[1];
        } else {
          raw.k[i][0] = *reinterpret_cast<const uint32_t*>(kslice + off);
        }
      } else {
        if constexpr (DPL == 8) {
          const u32x4 kk = *reinterpret_cast<const u32x4*>(kslice + off);
#pragma unroll
          for (int e = 0; e < 4; ++e) raw.k[i][e] = kk[e];
        } else {
          const u32x2 kk = *reinterpret_cast<const u32x2*>(kslice + off);
          raw.k[i][0] = kk[0]; raw.k[i][1] = kk[1];
        }
      }
    }
#pragma unroll
    for (int e = 0; e < DPL; ++e) {
      const int64_t off = (int64_t)((sub * DPL + e) * 16 + grp * TB) * C::kGElem;
      if constexpr (VW == 2) {
        const u32x2 vv = *reinterpret_cast<const u32x2*>(vslice + off);
        raw.v[e][0] = vv[0]; raw.v[e][1] = vv[1];
      } else {
        raw.v[e][0] = *reinterpret_cast<const uint32_t*>(vslice + off);
      }
    }
  };
  // packed bf16 pairs of a raw token vector
  auto pairs = [&](const raw_t& r, uint32_t (&o)[NP]) {
    if constexpr (FP8) {
#pragma unroll
      for (int q = 0; q < DPL / 4; ++q) {
        const f32x2 lo = __builtin_amdgcn_cvt_pk_f32_fp8(r[q], false);
        const f32x2 hi = __builtin_amdgcn_cvt_pk_f32_fp8(r[q], true);
        o[2 * q] = (__float_as_uint(lo[0]) >> 16) | (__float_as_uint(lo[1]) & 0xFFFF0000u);
        o[2 * q + 1] = (__float_as_uint(hi[0]) >> 16) | (__float_as_uint(hi[1]) & 0xFFFF0000u);
      }
    } else {
#pragma unroll
      for (int q = 0; q < NP; ++q) o[q] = r[q];
    }
  };

  uint32_t qp[RWS][NP];
  float o[RWS][DPL];
  float m_run[RWS], l_run[RWS];
  int nrows = 0;

  auto begin_item = [&](const int32_t* d) {
    nrows = uniform(d[IT_NROWS]);
#pragma unroll
    for (int row = 0; row < RWS; ++row) {
      int fork = 0, h = 0;
      item_row(plan, d, row, &fork, &h);
      const bool ok = row < nrows;
      // unconditional loads (padded rows read row 0 and are zeroed)
      const uint16_t* qrow = a.q + (ok ? ((int64_t)fork * plan.Hq + h) * D : 0) + sub * DPL;
#pragma unroll
      for (int q = 0; q < NP; ++q) {
        const uint32_t v = *reinterpret_cast<const uint32_t*>(qrow + 2 * q);
        qp[row][q] = ok ? v : 0u;
      }
      m_run[row] = -INFINITY;
      l_run[row] = 0.f;
#pragma unroll
      for (int e = 0; e < DPL; ++e) o[row][e] = 0.f;
    }
    wait_vmem();
  };

  auto compute_tile = [&](const Raw& raw, const int32_t* d, int r) {
    const int tile_in_item = uniform(d[IT_TILE0]) + (r - uniform(d[IT_RTILE0]));
    const int nv = uniform(d[IT_NVALID]);
    const int tok0 = tile_in_item * C::kTT + wave * 16 + grp * TB;   // first token of this stream
    uint32_t kp[TB][NP];
    float vf[TB][DPL];
#pragma unroll
    for (int i = 0; i < TB; ++i) pairs(raw.k[i], kp[i]);
#pragma unroll
    for (int e = 0; e < DPL; ++e) {
      if constexpr (FP8) {   // exact E4M3 decode of the TB tokens of dim e
        const f32x2 lo = __builtin_amdgcn_cvt_pk_f32_fp8(raw.v[e][0], false);
        const f32x2 hi = __builtin_amdgcn_cvt_pk_f32_fp8(raw.v[e][0], true);
        vf[0][e] = lo[0]; vf[1][e] = lo[1]; vf[2][e] = hi[0]; vf[3][e] = hi[1];
      } else {
#pragma unroll
        for (int i = 0; i < TB; ++i) vf[i][e] = __uint_as_float((raw.v[e][i >> 1] >> (16 * (i & 1))) << 16);
      }
    }
    // values of tokens past the item's end may be any bits, NaN included
#pragma unroll
    for (int i = 0; i < TB; ++i)
      if (tok0 + i >= nv) {
#pragma unroll
        for (int e = 0; e < DPL; ++e) vf[i][e] = 0.f;
      }
    float ksc = 1.f, vsc = 1.f;
    if constexpr (FP8) {
      ksc = scales[r * C::kIdsPerTile + wave];
      vsc = scales[C::kIdCap + r * C::kIdsPerTile + wave];
    }
#pragma unroll
    for (int row = 0; row < RWS; ++row) {
      if (row >= nrows) break;
      float s[TB];
#pragma unroll
      for (int i = 0; i < TB; ++i) {
        float acc = 0.f;
#pragma unroll
        for (int q = 0; q < NP; ++q)
          acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, qp[row][q]),
                                                __builtin_bit_cast(bf16x2, kp[i][q]),
                                                acc, false);
        acc += __shfl_xor(acc, 1, 64);
        acc += __shfl_xor(acc, 2, 64);
        acc += __shfl_xor(acc, 4, 64);
        acc += __shfl_xor(acc, 8, 64);
        s[i] = (tok0 + i < nv) ? acc * ksc : -INFINITY;
      }
      const float mx = fmaxf(fmaxf(s[0], s[1]), fmaxf(s[2], s[3]));
      const float m_new = fmaxf(m_run[row], mx);
      const float mc = (m_new == -INFINITY) ? 0.f : m_new * a.c_log2;
      const float alpha = __builtin_amdgcn_exp2f(m_run[row] * a.c_log2 - mc);
      m_run[row] = m_new;
      float p[TB];
      float ps = 0.f;
#pragma unroll
      for (int i = 0; i < TB; ++i) {
        p[i] = __builtin_amdgcn_exp2f(fmaf(s[i], a.c_log2, -mc));
        ps += p[i];
      }
      l_run[row] = l_run[row] * alpha + ps;
#pragma unroll
      for (int e = 0; e < DPL; ++e) {
        float acc = o[row][e] * alpha;
#pragma unroll
        for (int i = 0; i < TB; ++i) acc = fmaf(p[i] * vsc, vf[i][e], acc);
        o[row][e] = acc;
      }
    }
  };

  float* comb = reinterpret_cast<float*>(lds + C::kOffComb);
  float* comb_m = reinterpret_cast<float*>(lds + C::kOffML);
  float* comb_l = comb_m + 4 * RWS;
  auto finish_item = [&](const int32_t* d) {
    // combine the four streams of the wave (lanes sub, sub^16, sub^32, sub^48)
#pragma unroll
    for (int row = 0; row < RWS; ++row) {
      if (row >= nrows) break;
#pragma unroll
      for (int msk = 16; msk <= 32; msk <<= 1) {
        const float mo = __shfl_xor(m_run[row], msk, 64);
        const float lo = __shfl_xor(l_run[row], msk, 64);
        const float m = fmaxf(m_run[row], mo);
        const float mc = (m == -INFINITY) ? 0.f : m * a.c_log2;
        const float a0 = __builtin_amdgcn_exp2f(m_run[row] * a.c_log2 - mc);
        const float a1 = __builtin_amdgcn_exp2f(mo * a.c_log2 - mc);
#pragma unroll
        for (int e = 0; e < DPL; ++e) {
          const float oo = __shfl_xor(o[row][e], msk, 64);
          o[row][e] = o[row][e] * a0 + oo * a1;
        }
        l_run[row] = l_run[row] * a0 + lo * a1;
        m_run[row] = m;
      }
      if (grp == 0) {
#pragma unroll
        for (int e = 0; e < DPL; ++e) comb[(wave * RWS + row) * D + sub * DPL + e] = o[row][e];
        if (sub == 0) {
          comb_m[wave * RWS + row] = m_run[row];
          comb_l[wave * RWS + row] = l_run[row];
        }
      }
    }
    lds_barrier();
    // combine the four waves: thread -> (row, 8 or 4 dims)
    {
      constexpr int PER = RWS * D / C::kThreads;   // 8 (D=128) or 4 (D=64)
      const int row = tid / (D / PER);
      const int d0 = (tid % (D / PER)) * PER;
      const bool live = row < nrows;
      float m = -INFINITY, l = 0.f, acc[PER];
#pragma unroll
      for (int e = 0; e < PER; ++e) acc[e] = 0.f;
      if (live) {
#pragma unroll
        for (int wv = 0; wv < 4; ++wv) m = fmaxf(m, comb_m[wv * RWS + row]);
        const float mc = (m == -INFINITY) ? 0.f : m * a.c_log2;
#pragma unroll
        for (int wv = 0; wv < 4; ++wv) {
          const float sc = __builtin_amdgcn_exp2f(comb_m[wv * RWS + row] * a.c_log2 - mc);
          l += comb_l[wv * RWS + row] * sc;
#pragma unroll
          for (int e = 0; e < PER; ++e) acc[e] += comb[(wv * RWS + row) * D + d0 + e] * sc;
        }
      }
      // the row's largest |o| sets its fp16 scale (its D / PER threads are
      // consecutive lanes)
      float amax = 0.f;
#pragma unroll
      for (int e = 0; e < PER; ++e) amax = fmaxf(amax, fabsf(acc[e]));
#pragma unroll
      for (int o = 1; o < D / PER; o <<= 1) amax = fmaxf(amax, __shfl_xor(amax, o, 64));
      if (live) {
        const int k = uniform(d[IT_ORD]) - wr.first_ord;
        const int64_t slot = slot_of(pp, w, k);
        if (slot >= 0) {
          const float inv_l = 1.f / l;
          const uint32_t kexp = (uint32_t)part_row_k(__float_as_uint(amax * inv_l));
          const float mul = inv_l * __uint_as_float((254u - kexp) << 23);
          uint32_t* op = reinterpret_cast<uint32_t*>(a.ws + part_o_off(pp, slot, row, D)) + d0 / 2;
          if constexpr (PER == 8) {
            *reinterpret_cast<u32x4*>(op) = u32x4{pack_f16x2(acc[0] * mul, acc[1] * mul), pack_f16x2(acc[2] * mul, acc[3] * mul),
                                                  pack_f16x2(acc[4] * mul, acc[5] * mul), pack_f16x2(acc[6] * mul, acc[7] * mul)};
          } else {
            static_assert(PER == 4, "4 or 8 dims per thread");
            *reinterpret_cast<u32x2*>(op) = u32x2{pack_f16x2(acc[0] * mul, acc[1] * mul), pack_f16x2(acc[2] * mul, acc[3] * mul)};
          }
          if (d0 == 0)
            *reinterpret_cast<f32x2*>(a.ws + part_l_off(pp, slot, row)) =
                f32x2{m * a.sm_scale + __logf(l), __uint_as_float(kexp << 23)};
        }
      }
    }
    lds_barrier();
  };

  Raw cur, nxt;
  load_tile(cur, 0);
  int cur_item = -1;
  for (int r = 0; r < R; ++r) {
    load_tile(nxt, r + 1);
    const int ii = uniform(item_of_tile(items, nitems, r));
    const int32_t* d = items + ii * kItemInts;
    if (ii != cur_item) {
      begin_item(d);
      cur_item = ii;
    }
    compute_tile(cur, d, r);
    if (r - uniform(d[IT_RTILE0]) == uniform(d[IT_NTILE]) - 1) finish_item(d);
    cur = nxt;
  }
}

template <int D, bool FP8>
hipError_t launch_attn_dot_t(const AttnArgs& a, const Plan& plan, hipStream_t stream) {
  const int W = plan.part[kPartDot].workers;
  if (W <= 0) return hipSuccess;
  hipLaunchKernelGGL((attn_dot_kernel<D, FP8>), dim3(W), dim3(256), 0, stream, a, plan);
  return hipGetLastError();
}

hipError_t launch_attn_dot_any(const AttnArgs& a, const Plan& plan, bool fp8, hipStream_t stream) {
  if (plan.D == 128) return fp8 ? launch_attn_dot_t<128, true>(a, plan, stream) : launch_attn_dot_t<128, false>(a, plan, stream);
  return fp8 ? launch_attn_dot_t<64, true>(a, plan, stream) : launch_attn_dot_t<64, false>(a, plan, stream);
}

int dot_tile_tokens(int) { return DotCfg<128, false>::kTT; }
int dot_rows() { return DotCfg<128, false>::kRows; }
int dot_item_cap() { return DotCfg<128, false>::kItemCap; }
int dot_tile_cap(int) { return DotCfg<128, false>::kTileCap; }

}  // namespace specgen
