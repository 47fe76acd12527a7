// merge.h -- the log-sum-exp merge of one output row of fork-decode attention
// from the partial results the split attention kernels left in the workspace
// (used by the merge kernel, merge.hip).
//
// Partials over disjoint key sets combine exactly: with M = max_s lse_s and
// w_s = exp(lse_s - M), out = sum_s w_s o_s / sum_s w_s and
// lse = M + ln sum_s w_s (a part with lse = -inf is empty and is skipped).
#pragma once
#include "common.h"
#include "plan.h"

namespace specgen {

// Row merge for D in {64, 128} over partial rows stored as fp16 with a
// per-row power-of-two scale (plan.h, part_row_k): lanes read 16 bytes (8
// dims) each, so one load instruction covers PPI = 64 / (D/8) parts.  A batch
// is up to 64 parts: each lane loads one part's (lse, dec) pair and the wave
// issues the o loads of every part of the batch before it waits for any of
// them, so a row of up to 64 parts costs one memory round trip.
template <int D, typename PO, typename PL>
__device__ __forceinline__ void merge_row_v4(int nparts, PO part_o, PL part_ld, uint16_t* out_row,
                                             float* out_lse_p) {
  constexpr int LPP = D / 8;       // lanes per part
  constexpr int PPI = 64 / LPP;    // parts per load instruction
  constexpr int U = 64 / PPI;      // load instructions per batch
  constexpr int kBatch = PPI * U;  // parts per batch: one (lse, dec) per lane
  static_assert(kBatch == 64 && (LPP == 16 || LPP == 8), "one part per lane; lane groups of 16 or 8");
  const int lane = threadIdx.x & 63;
  const int gsl = lane / LPP;      // part slot of this lane within an instruction
  const int c8 = (lane % LPP) * 8; // first of the 8 dims this lane owns
  float M = -INFINITY, z = 0.f;
  float acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.f;
  for (int p0 = 0; p0 < nparts; p0 += kBatch) {
    const int cnt = (nparts - p0) < kBatch ? (nparts - p0) : kBatch;
    const f32x2 ld = lane < cnt ? part_ld(p0 + lane) : f32x2{-INFINITY, 0.f};
    const float l = ld[0];
    u32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      v[u] = u32x4{0u, 0u, 0u, 0u};
      if (u * PPI < cnt) {   // wave-uniform: only instructions that hold a part
        const int q = u * PPI + gsl;
        const int qc = q < cnt ? q : cnt - 1;   // the last instruction's spare slots re-read its last part
        v[u] = *reinterpret_cast<const u32x4*>(part_o(p0 + qc) + c8 / 2);
      }
    }
    const float Mn = fmaxf(M, rows4_max(row16_max(l)));
    if (Mn == -INFINITY) continue;          // every part so far empty (wave-uniform)
    const float rescale = __expf(M - Mn);   // M = -inf -> 0
    z *= rescale;
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] *= rescale;
    M = Mn;
    const float wl = (l == -INFINITY) ? 0.f : __expf(l - M);
    z += rows4_sum(row16_sum(wl));
    const float wo = wl * ld[1];            // the weight of the stored (scaled) values
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int q = u * PPI + gsl;
      float wq = __shfl(wo, q < 64 ? q : 63, 64);
      if (q >= cnt) wq = 0.f;
      if (wq != 0.f) {   // an empty part's o may be garbage
#pragma unroll
        for (int h = 0; h < 4; ++h) {
          const f32x2 x = unpack_f16x2(v[u][h]);
          acc[2 * h] = fmaf(wq, x[0], acc[2 * h]);
          acc[2 * h + 1] = fmaf(wq, x[1], acc[2 * h + 1]);
        }
      }
    }
  }
  // sum the PPI lane groups: the four 16-lane rows (D = 128), or the eight
  // 8-lane halves of rows (D = 64)
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    if constexpr (LPP == 8) acc[e] = xor8_sum(acc[e]);
    acc[e] = rows4_sum(acc[e]);
  }
  const bool empty = (M == -INFINITY);
  if (gsl == 0) {
    const float inv = empty ? 0.f : 1.f / z;
    u32x4 pk;
#pragma unroll
    for (int h = 0; h < 4; ++h) pk[h] = pack_bf16x2(empty ? 0.f : acc[2 * h] * inv, empty ? 0.f : acc[2 * h + 1] * inv);
    *reinterpret_cast<u32x4*>(out_row + c8) = pk;
  }
  if (out_lse_p && lane == 0) *out_lse_p = empty ? -INFINITY : M + __logf(z);
}

// The row (f, h) = (row / Hq, row % Hq) of the output: the parts are the
// partials of the workers that covered its prefix item and its suffix item.
// One wavefront per row; `plan` may live in LDS or in the kernel arguments.
template <int D>
__device__ __forceinline__ void fork_merge_row(const Plan& plan, const float* __restrict__ ws, int64_t row,
                                               uint16_t* __restrict__ out, float* __restrict__ out_lse) {
  const int f = (int)(row / plan.Hq);
  const int h = (int)(row % plan.Hq);
  // The item table (written by the partial kernels' walks) gives each item's
  // first and last worker and its segment index in the first one.  Part i of
  // an item sits in slot (w_lo + i) * kmax + (i == 0 ? k_lo : 0), so relative
  // to part 0 it is i * kmax - k_lo slots further (plain scalars: a lane picks
  // the prefix or the suffix item by its part index).
  int Xs[2] = {0, 0}, ords[2] = {0, 0}, rs[2] = {0, 0};
  bool has[2];
  prefix_item_of_row(plan, f, h, &Xs[0], &ords[0], &rs[0]);
  has[0] = true;
  has[1] = suffix_item_of_row(plan, f, h, &Xs[1], &ords[1], &rs[1]);
  // both table entries are loaded before either is used
  int32_t e[2][3];
#pragma unroll
  for (int s2 = 0; s2 < 2; ++s2) {
    const int32_t* info = reinterpret_cast<const int32_t*>(ws + plan.part[Xs[s2]].info_base) + 3 * (int64_t)ords[s2];
#pragma unroll
    for (int c = 0; c < 3; ++c) e[s2][c] = has[s2] ? info[c] : 0;
  }
  int64_t o0[2] = {0, 0}, l0[2] = {0, 0};
  int kmax[2] = {1, 1}, klo[2] = {0, 0}, n[2] = {0, 0}, srows[2] = {1, 1};
  bool ok = true;
#pragma unroll
  for (int s2 = 0; s2 < 2; ++s2) {
    if (!has[s2]) continue;
    const int X = Xs[s2], ord = ords[s2], r = rs[s2];
    const PartPlan& pp = plan.part[X];
    const int w_lo = e[s2][0], w_hi = e[s2][1], k_lo = e[s2][2];
    if (ord < 0 || ord >= pp.n_items || w_lo < 0 || w_hi < w_lo || w_hi >= pp.workers || k_lo < 0 || k_lo >= pp.kmax) {
      ok = false;
      continue;
    }
    const int64_t slot0 = (int64_t)w_lo * pp.kmax + k_lo;
    o0[s2] = part_o_off(pp, slot0, r, D);
    l0[s2] = part_l_off(pp, slot0, r);
    kmax[s2] = pp.kmax;
    klo[s2] = k_lo;
    n[s2] = w_hi - w_lo + 1;
    srows[s2] = pp.slot_rows;
  }
  if (!ok) {   // the item table is inconsistent: fail loudly rather than read out of range
    const int lane = threadIdx.x & 63;
    for (int d = lane; d < D; d += 64) out[row * D + d] = 0x7FC0;   // bf16 NaN
    if (out_lse && lane == 0) out_lse[row] = __builtin_nanf("");
    return;
  }
  const int np = n[0];
  const int64_t pO0 = o0[0], sO0 = o0[1], pL0 = l0[0], sL0 = l0[1];
  const int pK = kmax[0], sK = kmax[1], pKlo = klo[0], sKlo = klo[1], pR = srows[0], sR = srows[1];
  auto rel_slots = [&](int p) -> int64_t {   // slots between part p and its item's part 0
    const bool pre = p < np;
    const int i = pre ? p : p - np;
    return i == 0 ? 0 : (int64_t)i * (pre ? pK : sK) - (pre ? pKlo : sKlo);
  };
  auto po = [&](int p) {   // the part's o row: D fp16 values, two per uint32
    const bool pre = p < np;
    return reinterpret_cast<const uint32_t*>(ws + (pre ? pO0 : sO0) + rel_slots(p) * (int64_t)(pre ? pR : sR) * (D / 2));
  };
  auto pl = [&](int p) {   // its (lse, dec) pair
    const bool pre = p < np;
    return *reinterpret_cast<const f32x2*>(ws + (pre ? pL0 : sL0) + rel_slots(p) * (int64_t)(pre ? pR : sR) * 2);
  };
  merge_row_v4<D>(np + n[1], po, pl, out + row * D, out_lse ? out_lse + row : nullptr);
}

}  // namespace specgen
