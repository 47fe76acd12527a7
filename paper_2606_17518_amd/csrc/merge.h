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
// is U load instructions, PPI * U parts (at most 64): each lane loads one
// part's (lse, dec) pair and the wave issues the o loads of every part of the
// batch before it waits for any of them, so a row of up to PPI * U parts costs
// one memory round trip.  The o registers of a batch set the kernel's register
// count, and with it how many waves a compute unit holds, so the launch takes
// the smallest U that covers the plan's rows.
template <int D, int U, typename PO, typename PL>
__device__ __forceinline__ void merge_row_v4(int nparts, PO part_o, PL part_ld, uint16_t* out_row,
                                             float* out_lse_p) {
  constexpr int LPP = D / 8;       // lanes per part
  constexpr int PPI = 64 / LPP;    // parts per load instruction
  constexpr int kBatch = PPI * U;  // parts per batch: one (lse, dec) per lane
  static_assert(kBatch <= 64 && (LPP == 16 || LPP == 8), "at most one part per lane; lane groups of 16 or 8");
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
// partials of the workers that covered its prefix items (one per trace on the
// fork's prefix chain: its own trace and, with nested prefixes, each ancestor)
// and its suffix item.  kDepth bounds the chain (1: no nesting).  One
// wavefront per row; `plan` may live in LDS or in the kernel arguments.
struct MergeLoc {
  int64_t slots;   // slots between a part and its item's part 0
  int64_t o, l;    // the item's part-0 offsets
  int rows;
};
struct alignas(16) MergeItemLoc {
  int64_t o, l;
  int kmax, klo, rows, first;
};

// loc: kDepth + 1 entries of LDS private to the calling wavefront (unused
// when kDepth == 1).
template <int D, int kDepth, int kU>
__device__ __forceinline__ void fork_merge_row(const Plan& plan, const float* __restrict__ ws, int64_t row,
                                               uint16_t* __restrict__ out, float* __restrict__ out_lse,
                                               MergeItemLoc* loc) {
  constexpr int kItems = kDepth + 1;   // prefix items nearest trace first, then the suffix item
  const int f = (int)(row / plan.Hq);
  const int h = (int)(row % plan.Hq);
  // The item table (written by the partial kernels' walks) gives each item's
  // first and last worker and its segment index in the first one.  Part i of
  // an item sits in slot (w_lo + i) * kmax + (i == 0 ? k_lo : 0), so relative
  // to part 0 it is i * kmax - k_lo slots further (plain scalars: a lane picks
  // its part's item by the part index).
  int Xs[kItems], ords[kItems], rs[kItems];
  bool has[kItems];
  int t = trace_of_fork(plan, f);
#pragma unroll
  for (int i = 0; i < kDepth; ++i) {
    Xs[i] = ords[i] = rs[i] = 0;
    has[i] = t >= 0;
    if (has[i]) {
      prefix_item_of_row(plan, f, h, t, &Xs[i], &ords[i], &rs[i]);
      t = plan.parent[t];
    }
  }
  Xs[kDepth] = ords[kDepth] = rs[kDepth] = 0;
  has[kDepth] = suffix_item_of_row(plan, f, h, &Xs[kDepth], &ords[kDepth], &rs[kDepth]);
  // every table entry is loaded before any is used
  int32_t e[kItems][3];
#pragma unroll
  for (int s2 = 0; s2 < kItems; ++s2) {
    const int32_t* info = reinterpret_cast<const int32_t*>(ws + plan.part[Xs[s2]].info_base) + 3 * (int64_t)ords[s2];
#pragma unroll
    for (int c = 0; c < 3; ++c) e[s2][c] = has[s2] ? info[c] : 0;
  }
  int64_t o0[kItems], l0[kItems];
  int kmax[kItems], klo[kItems], first[kItems + 1], srows[kItems];
  bool ok = true;
  first[0] = 0;
#pragma unroll
  for (int s2 = 0; s2 < kItems; ++s2) {
    o0[s2] = l0[s2] = 0;
    kmax[s2] = srows[s2] = 1;
    klo[s2] = 0;
    int n = 0;
    if (has[s2]) {
      const int X = Xs[s2], ord = ords[s2], r = rs[s2];
      const PartPlan& pp = plan.part[X];
      const int w_lo = e[s2][0], w_hi = e[s2][1], k_lo = e[s2][2];
      if (ord < 0 || ord >= pp.n_items || w_lo < 0 || w_hi < w_lo || w_hi >= pp.workers || k_lo < 0 ||
          k_lo >= pp.kmax) {
        ok = false;
      } else {
        const int64_t slot0 = (int64_t)w_lo * pp.kmax + k_lo;
        o0[s2] = part_o_off(pp, slot0, r, D);
        l0[s2] = part_l_off(pp, slot0, r);
        kmax[s2] = pp.kmax;
        klo[s2] = k_lo;
        n = w_hi - w_lo + 1;
        srows[s2] = pp.slot_rows;
      }
    }
    first[s2 + 1] = first[s2] + n;   // an absent item holds no parts
  }
  if (!ok) {   // the item table is inconsistent: fail loudly rather than read out of range
    const int lane = threadIdx.x & 63;
    for (int d = lane; d < D; d += 64) out[row * D + d] = 0x7FC0;   // bf16 NaN
    if (out_lse && lane == 0) out_lse[row] = __builtin_nanf("");
    return;
  }
  // Picking a part's item: with one prefix item, per-lane selects between
  // named scalars; with a chain, the wave's item table in LDS (`loc`, kItems
  // entries), indexed by the number of items that start at or before the
  // part.  (Selecting between elements of a register array would make the
  // compiler index the array in private memory instead.)
  const int64_t pO = o0[0], pL = l0[0], sO = o0[kItems - 1], sL = l0[kItems - 1];
  const int pK = kmax[0], pKlo = klo[0], pR = srows[0], sK = kmax[kItems - 1], sKlo = klo[kItems - 1],
            sR = srows[kItems - 1], np = first[1];
  if constexpr (kItems > 2) {
    if ((threadIdx.x & 63) == 0) {
#pragma unroll
      for (int s2 = 0; s2 < kItems; ++s2) loc[s2] = MergeItemLoc{o0[s2], l0[s2], kmax[s2], klo[s2], srows[s2], first[s2]};
    }
    __builtin_amdgcn_wave_barrier();
  }
  auto locate_part = [&](int p) {   // the last item whose first part is <= p owns p
    if constexpr (kItems == 2) {
      const bool pre = p < np;
      const int i = pre ? p : p - np;
      const int K = pre ? pK : sK, KL = pre ? pKlo : sKlo;
      return MergeLoc{i == 0 ? 0 : (int64_t)i * K - KL, pre ? pO : sO, pre ? pL : sL, pre ? pR : sR};
    } else {
      int k = 0;
#pragma unroll
      for (int s2 = 1; s2 < kItems; ++s2) k += p >= first[s2];
      const MergeItemLoc it = loc[k];
      const int i = p - it.first;
      return MergeLoc{i == 0 ? 0 : (int64_t)i * it.kmax - it.klo, it.o, it.l, it.rows};
    }
  };
  auto po = [&](int p) {   // the part's o row: D fp16 values, two per uint32
    const MergeLoc L = locate_part(p);
    return reinterpret_cast<const uint32_t*>(ws + L.o + L.slots * (int64_t)L.rows * (D / 2));
  };
  auto pl = [&](int p) {   // its (lse, dec) pair
    const MergeLoc L = locate_part(p);
    return *reinterpret_cast<const f32x2*>(ws + L.l + L.slots * (int64_t)L.rows * 2);
  };
  merge_row_v4<D, kU>(first[kItems], po, pl, out + row * D, out_lse ? out_lse + row : nullptr);
}

// Several rows per wave: one row per group of D/8 lanes -- four rows per wave
// at D = 128, eight at D = 64 -- each lane holding 8 dims of its row.  A row's
// item table entries take one memory round trip and its parts one more per
// batch of kParts, and a wave carries four or eight rows through them at once,
// where the one-row-per-wave merge leaves most lanes idle on rows of a handful
// of parts and holds fewer rows in flight.  kDepth <= 2 (the per-lane item
// selection below is a pair of comparisons).
template <int D, int kDepth, int kParts>
__device__ __forceinline__ void fork_merge_rows_grouped(const Plan& plan, const float* __restrict__ ws, int64_t row,
                                                        uint16_t* __restrict__ out, float* __restrict__ out_lse) {
  static_assert(kDepth <= 2, "per-lane item selection covers a prefix chain of at most two traces");
  constexpr int LPP = D / 8;           // lanes per row
  constexpr int kItems = kDepth + 1;   // prefix items nearest trace first, then the suffix item
  const int lane = threadIdx.x & 63;
  const int c8 = (lane % LPP) * 8;     // first of the 8 dims this lane owns
  const bool live = row < (int64_t)plan.N * plan.Hq;
  const int64_t rw = live ? row : 0;   // the spare groups of a last wave read row 0 and store nothing
  const int f = (int)(rw / plan.Hq);
  const int h = (int)(rw % plan.Hq);
  int Xs[kItems], ords[kItems], rs[kItems];
  bool has[kItems];
  int t = trace_of_fork(plan, f);
#pragma unroll
  for (int i = 0; i < kDepth; ++i) {
    Xs[i] = ords[i] = rs[i] = 0;
    has[i] = t >= 0;
    if (has[i]) {
      prefix_item_of_row(plan, f, h, t, &Xs[i], &ords[i], &rs[i]);
      t = plan.parent[t];
    }
  }
  Xs[kDepth] = ords[kDepth] = rs[kDepth] = 0;
  has[kDepth] = suffix_item_of_row(plan, f, h, &Xs[kDepth], &ords[kDepth], &rs[kDepth]);
  int32_t e[kItems][3];
#pragma unroll
  for (int s2 = 0; s2 < kItems; ++s2) {
    const int32_t* info = reinterpret_cast<const int32_t*>(ws + plan.part[Xs[s2]].info_base) + 3 * (int64_t)ords[s2];
#pragma unroll
    for (int c = 0; c < 3; ++c) e[s2][c] = has[s2] ? info[c] : 0;
  }
  int64_t o0[kItems], l0[kItems];
  int kmax[kItems], klo[kItems], first[kItems + 1], srows[kItems];
  bool ok = true;
  first[0] = 0;
#pragma unroll
  for (int s2 = 0; s2 < kItems; ++s2) {
    o0[s2] = l0[s2] = 0;
    kmax[s2] = srows[s2] = 1;
    klo[s2] = 0;
    int n = 0;
    if (has[s2]) {
      const PartPlan& pp = plan.part[Xs[s2]];
      const int w_lo = e[s2][0], w_hi = e[s2][1], k_lo = e[s2][2];
      if (ords[s2] < 0 || ords[s2] >= pp.n_items || w_lo < 0 || w_hi < w_lo || w_hi >= pp.workers || k_lo < 0 ||
          k_lo >= pp.kmax) {
        ok = false;
      } else {
        const int64_t slot0 = (int64_t)w_lo * pp.kmax + k_lo;
        o0[s2] = part_o_off(pp, slot0, rs[s2], D);
        l0[s2] = part_l_off(pp, slot0, rs[s2]);
        kmax[s2] = pp.kmax;
        klo[s2] = k_lo;
        n = w_hi - w_lo + 1;
        srows[s2] = pp.slot_rows;
      }
    }
    first[s2 + 1] = first[s2] + n;
  }
  const int np = first[kItems];
  if (!ok) {   // the item table is inconsistent: fail loudly rather than read out of range
    if (live) {
      *reinterpret_cast<u32x4*>(out + row * D + c8) = u32x4{0x7FC07FC0u, 0x7FC07FC0u, 0x7FC07FC0u, 0x7FC07FC0u};
      if (out_lse && lane % LPP == 0) out_lse[row] = __builtin_nanf("");
    }
    return;
  }
  float M = -INFINITY, z = 0.f, acc[8];
#pragma unroll
  for (int q = 0; q < 8; ++q) acc[q] = 0.f;
  // batches of kParts parts: every part's (lse, dec) and this lane's 8 dims of
  // its o loaded before any is used; running max and sums carried across batches
  for (int p0 = 0; p0 < np; p0 += kParts) {
    f32x2 ld[kParts];
    u32x4 v[kParts];
#pragma unroll
    for (int pi = 0; pi < kParts; ++pi) {
      const int p = p0 + pi;
      ld[pi] = f32x2{-INFINITY, 0.f};
      v[pi] = u32x4{0u, 0u, 0u, 0u};
      if (p < np) {
        const int s2 = kItems == 2 ? (p >= first[1] ? 1 : 0) : (p >= first[2] ? 2 : (p >= first[1] ? 1 : 0));
        const int i = p - (s2 == 0 ? 0 : s2 == 1 ? first[1] : first[kItems - 1]);
        const int K = s2 == 0 ? kmax[0] : s2 == 1 ? kmax[1] : kmax[kItems - 1];
        const int KL = s2 == 0 ? klo[0] : s2 == 1 ? klo[1] : klo[kItems - 1];
        const int R = s2 == 0 ? srows[0] : s2 == 1 ? srows[1] : srows[kItems - 1];
        const int64_t O = s2 == 0 ? o0[0] : s2 == 1 ? o0[1] : o0[kItems - 1];
        const int64_t L = s2 == 0 ? l0[0] : s2 == 1 ? l0[1] : l0[kItems - 1];
        const int64_t slots = i == 0 ? 0 : (int64_t)i * K - KL;
        ld[pi] = *reinterpret_cast<const f32x2*>(ws + L + slots * R * 2);
        v[pi] = *reinterpret_cast<const u32x4*>(
            reinterpret_cast<const uint32_t*>(ws + O + slots * (int64_t)R * (D / 2)) + c8 / 2);
      }
    }
    float Mn = M;
#pragma unroll
    for (int pi = 0; pi < kParts; ++pi) Mn = fmaxf(Mn, ld[pi][0]);
    if (Mn == -INFINITY) continue;   // every part so far empty
    const float rescale = __expf(M - Mn);   // M = -inf -> 0
    z *= rescale;
#pragma unroll
    for (int q = 0; q < 8; ++q) acc[q] *= rescale;
    M = Mn;
#pragma unroll
    for (int pi = 0; pi < kParts; ++pi) {
      const float w = ld[pi][0] == -INFINITY ? 0.f : __expf(ld[pi][0] - M);
      z += w;
      const float wo = w * ld[pi][1];   // the weight of the stored (scaled) values
      if (wo != 0.f) {                  // an empty part's o may be garbage
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const f32x2 x = unpack_f16x2(v[pi][q]);
          acc[2 * q] = fmaf(wo, x[0], acc[2 * q]);
          acc[2 * q + 1] = fmaf(wo, x[1], acc[2 * q + 1]);
        }
      }
    }
  }
  if (!live) return;
  const bool empty = M == -INFINITY;
  const float inv = empty ? 0.f : 1.f / z;
  u32x4 pk;
#pragma unroll
  for (int q = 0; q < 4; ++q) pk[q] = pack_bf16x2(acc[2 * q] * inv, acc[2 * q + 1] * inv);
  *reinterpret_cast<u32x4*>(out + row * D + c8) = pk;
  if (out_lse && lane % LPP == 0) out_lse[row] = empty ? -INFINITY : M + __logf(z);
}

}  // namespace specgen
