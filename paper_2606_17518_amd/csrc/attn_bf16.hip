// attn_bf16.hip -- the bf16 shared-prefix (and suffix) partial-attention
// kernel on gfx950 matrix cores: eight waves per workgroup, tiles streamed
// from HBM straight into LDS.
//
// One workgroup = one worker of the MFMA partition (plan.h).  It walks its
// range of work items; an item's rows are every (fork, q head) pair of a GQA
// group of one trace (prefix item: the trace's shared prefix is read from HBM
// once for all its forks, Sec. 4.2 / Sec. 8.7) or the g heads of one fork
// (suffix item).
//
// KV layout.  Inside a pool block, kv head j's K is 16 token rows of D values
// and its V is D rows of 16 token values (V transposed), each 16*D*2 bytes.
// A tile of TT tokens is TT/16 such block slices per tensor.
//
// Slots.  The worker's range is a sequence of 32 KiB slots: for each item one
// "q slot" per 128 query rows (128 x D bf16 each) followed by its tiles (TT
// tokens of K, then TT tokens of V).  Slots go through a ring of four LDS
// stages with three slots in flight.  Every wave moves the same number of
// 1 KiB pieces of every slot with global_load_lds_dwordx4 (64 lanes x 16 B, no
// VGPR staging; tiles nontemporal, the KV is read once; q slots through the
// caches, since every worker of a prefix item reads the same q rows): four of a
// bf16 slot (waves 0-3 the K block slices of a tile, waves 4-7 its V slices),
// two of an E4M3 tile (one of its K codes, one of its V codes).  So the number
// of vector-memory operations a wave has in flight is known exactly and the
// wait for slot s is "vmcnt <= (pieces per slot) x (slots issued after s) +
// partial stores issued since".  These
// loads are issued from inline asm: the compiler does not see them, so it
// neither drains them (vmcnt(0)) before LDS reads nor reorders them across
// the LDS barriers.
//
// Rows and tokens.  An item with r <= 256 rows uses RG = ceil(r / 32) row
// groups of 32 rows and splits each tile's tokens over TG = min(TT/32, 8/RG)
// token groups: wave w computes row group w % RG over token group w / RG (two
// token groups for the 128-row prefix items, the two waves of a SIMD, whose
// vector and matrix work can overlap when they do not run in step: the slot
// loop staggers their DMA issue for that; one token group for 5-8 row groups,
// where each wave runs both slabs of a tile).  An item of more than 128 rows has two q slots, and a
// wave reads its Q^T from the one holding its rows.  Items with fewer rows pad
// their last row group; they are bound by their K/V bytes, not by the matrix
// cores (one wave's dependent chain through a 32-token slab takes about 0.9
// us, so their tiles are split over two waves).  At the item's end the token
// groups are combined through the stage that was just consumed, and token
// group 0 writes the normalised partial (o, lse).
//
// Math per 32-token slab and 16-row N-tile: S^T = K Q^T on
// v_mfma_f32_16x16x32_bf16 (A = 16 keys x 32 dims from LDS, B = Q^T in
// VGPRs) with the keys of the two S^T tiles taken so that each lane's 8 scores
// are the 8 consecutive tokens the PV operand needs; online softmax in base 2
// with lazy rescaling; O^T += V^T P^T, where the A operand (16 dims x 32
// tokens) is one 16-byte LDS read per lane because V is stored transposed.
//
// E4M3 KV with fp8 scores (QK8): S^T = K Q^T runs on gfx950's fp8 matrix cores
// (v_mfma_scale_f32_16x16x128_f8f6f4: all 128 dims of 16 keys x 16 rows in one
// instruction) straight from the K codes in LDS, which are then never decoded;
// each query row is held as two E4M3 terms, q = 2^e (hi + lo / 16), whose
// power-of-two scale rides in the instruction's per-row E8M0 scale operand, so
// the score is the hi product accumulated onto the lo product.  A single E4M3
// term would double the score rate but moves peaked scores by several percent;
// with two terms the scores are as close as with bf16 queries at the same
// matrix time (the fp8 instruction runs at twice the bf16 rate).  The PV
// product stays on bf16 operands (V codes are decoded in LDS, and P in E4M3
// would be as coarse as a one-term query).
//
// The accumulators live in VGPRs: this file is compiled with MFMA operands and
// results in VGPRs (-amdgpu-mfma-vgpr-form), which leaves the whole 256-register
// budget of a two-waves-per-SIMD kernel to one register file.  It is also
// compiled without IEEE-mode NaN quieting (-mno-amdgpu-ieee -fno-honor-nans):
// the row maxima would otherwise cost three instructions per element.  Masked
// scores are -inf, never NaN, and infinities keep their meaning.
#include "worker.h"
#include "lds_layout.h"

namespace specgen {

#ifdef SPECGEN_TIMELINE
// Timeline build (libspecgen_timeline.so only): thread 0 of every workgroup
// stamps the GPU's constant 100 MHz clock at fixed points of its run into LDS
// (kernel start, plan in LDS, walk done, every slot landed, end) and wave 0
// writes the stamps out when the workgroup ends.  Nothing is stored to global
// memory inside the slot loop, so the DMA accounting of the ring is untouched;
// each stamp costs thread 0 a clock read.
constexpr int kTlWorkers = 2048;   // workgroups recorded
constexpr int kTlSlots = 128;      // 0 start, 1 plan, 2 walk, 3 first slots issued, 4 + s slot s landed, 127 end
__device__ uint64_t g_tl_stamp[kTlWorkers][kTlSlots];
__device__ int32_t g_tl_kind[kTlWorkers][kTlSlots];
#endif

namespace bf16k {

// l + the sum of the 8 bf16 probabilities packed in pk (one dot2 with (1, 1)
// per pair): the sum of exactly the weights the PV product uses.  The
// elements are copied to scalars first: __builtin_bit_cast applied to an
// element of an ext_vector_type value reads element 0 whatever the index.
__device__ __forceinline__ float row_sum_bf16(const u32x4 pk, float l) {
  const bf16x2 one = __builtin_bit_cast(bf16x2, 0x3F803F80u);
  const uint32_t w0 = pk.x, w1 = pk.y, w2 = pk.z, w3 = pk.w;
  float a0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w0), one, 0.f, false);
  float a1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w1), one, l, false);
  a0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w2), one, a0, false);
  a1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w3), one, a1, false);
  return a0 + a1;
}

// The running max moves only when a new score would give a probability above
// 2^kRescaleLog2 relative to it.
constexpr float kRescaleLog2 = 8.f;

template <int D, bool FP8>
struct Cfg {
  static constexpr int kThreads = 512;
  static constexpr int kWaves = 8;
  static constexpr int kTT = (D == 128) ? 64 : 128;   // tokens per tile
  static constexpr int kRowB = D * 2;                 // bytes per K (or q) row
  static constexpr int kCPR = kRowB / 16;             // 16-byte chunks per row
  static constexpr int kTileB = kTT * kRowB;          // K (or V) bytes of a tile: 16 KiB
  static constexpr int kSliceB = 16 * kRowB;          // one block's slice of one kv head and tensor
  static constexpr int kStageB = 2 * kTileB;          // one slot
  static constexpr int kStages = 4;
  static constexpr int kRPI = 1024 / kRowB;           // K rows moved by one wave instruction
  static constexpr int kDmaSlot = 4;                  // instructions per wave per slot
  static constexpr int kSlicesPerWave = kTT / 16 / 4; // block slices of a tile per wave (4 waves per tensor)
  static constexpr int kPiecesPerSlice = kSliceB / 1024;
  static constexpr int kItemCap = 64;
  static constexpr int kMaxRows = 256;                // rows per item (row block)
  static constexpr int kQRows = 128;                  // q rows per slot: an item takes 1 or 2 q slots
  static constexpr int kOffItems = kStages * kStageB;
  static constexpr int kOffML = kOffItems + kItemCap * kItemInts * 4;
  static constexpr int kMLBytes = kWaves * 2 * 16 * 4 * 4;   // [wave][nt][row] (m, l, lf, -)
  static constexpr int kOffIds = kOffML + kMLBytes;
  static constexpr int kIdCap = 2560;                 // block ids of a worker's range
  static constexpr int kIdsPerTile = kTT / 16;
  static constexpr int kTileCap = kIdCap / kIdsPerTile;
  // E4M3 KV: a tile slot lands 1 KiB pieces of K and V codes (two
  // instructions per wave instead of four), each at the start of the 2 KiB run
  // of the bf16 tile that its converting wave writes: K code piece n (64
  // chunks of 16 bytes: 8 token rows for D = 128, 16 for D = 64) fills bf16
  // K rows at 2 KiB * n, V code piece n the V^T rows at kTileB + 2 KiB * n.
  // Each wave then converts its own pieces in place, with no barrier.
  static constexpr int kF8Slice = 16 * D;             // code bytes of one block slice
  static constexpr int kTileDma = FP8 ? 2 : kDmaSlot; // instructions per wave of a tile slot
  static constexpr int kLdsBytes = kOffIds + kIdCap * 4;
  static_assert(kSlicesPerWave * kPiecesPerSlice == kDmaSlot, "a tile slot is four instructions per wave");
  static_assert(kDmaSlot * kWaves * 1024 == kStageB, "slot split over the waves");
  static_assert(kQRows * kRowB <= kStageB && 2 * kQRows >= kMaxRows, "q rows of an item fit two slots");
  static_assert(kLdsBytes + (int)sizeof(Plan) <= 163840, "LDS budget");
  static_assert(kMLBytes >= (2 * kWaves + 1) * 4, "the walk's scratch fits the ML area");
  static_assert(!FP8 || kSlicesPerWave * (kF8Slice / 1024) == kTileDma, "E4M3 code instructions per wave");
};

// q slots of an item of `nrows` rows (128 rows per slot)
__device__ __forceinline__ int q_slots(int nrows) { return nrows > 128 ? 2 : 1; }

// Chunk swizzle of the q rows in a slot: the 16 rows an MFMA operand read
// touches land in distinct banks.
template <int D>
__device__ __forceinline__ int swz_q(int row) { return D == 128 ? (row & 15) : ((row >> 1) & 7); }

// One wave instruction: 64 lanes x 16 bytes from gbase + voff (per lane) into
// LDS at lds_addr + 16 * lane, nontemporal.  gbase and lds_addr must be
// wave-uniform.  (The readfirstlanes only restate what holds: the compiler
// cannot always prove these operands uniform, and an SGPR operand must be.)
__device__ __forceinline__ void dma16(const void* gbase, uint32_t voff, uint32_t lds_addr) {
  const uint64_t g = reinterpret_cast<uint64_t>(gbase);
  const uint32_t glo = __builtin_amdgcn_readfirstlane((uint32_t)g);
  const uint32_t ghi = __builtin_amdgcn_readfirstlane((uint32_t)(g >> 32));
  const void* gu = reinterpret_cast<const void*>(((uint64_t)ghi << 32) | glo);
  const uint32_t l = __builtin_amdgcn_readfirstlane(lds_addr);
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1 nt" ::"v"(voff), "s"(gu), "s"(l) : "m0");
}

// The same, through the caches (for rows several workgroups read).
__device__ __forceinline__ void dma16_cached(const void* gbase, uint32_t voff, uint32_t lds_addr) {
  const uint64_t g = reinterpret_cast<uint64_t>(gbase);
  const uint32_t glo = __builtin_amdgcn_readfirstlane((uint32_t)g);
  const uint32_t ghi = __builtin_amdgcn_readfirstlane((uint32_t)(g >> 32));
  const void* gu = reinterpret_cast<const void*>(((uint64_t)ghi << 32) | glo);
  const uint32_t l = __builtin_amdgcn_readfirstlane(lds_addr);
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(gu), "s"(l) : "m0");
}

// Four E4M3 codes -> four bf16, one gfx950 scaled conversion per pair with
// scale 1: exact (every E4M3 value, NaN included, has a bf16 encoding).
__device__ __forceinline__ u32x2 e4m3x4_to_bf16x4(uint32_t w) {
  u32x2 r;
  r[0] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.f, false));
  r[1] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.f, true));
  return r;
}

typedef int i32x8 __attribute__((ext_vector_type(8)));

// fp8 scores: the XOR swizzle of the 16-byte chunks of K code row t (bit 0 from
// bit 1 of t, bits 1-2 from bits 3-4): the 16 rows an operand read touches in
// one lane group spread over all bank groups.
__device__ __forceinline__ int k8_swz(int t) { return ((t >> 1) & 1) | ((t >> 2) & 6); }

// The smallest e with amax * 2^-e <= 448 (E4M3's largest finite value), from
// the bits of amax, kept in [-123, 120] so that 127 + e and 127 + e - 4 are
// valid E8M0 scales and 2^-e is a normal float; 0 for a zero row.
__device__ __forceinline__ int q8_exponent(float amax) {
  const uint32_t b = __float_as_uint(amax);
  if (amax == 0.f) return 0;
  const int ex = (int)((b >> 23) & 0xFF) - 127;          // amax = 1.m x 2^ex
  int e = ex - 8 + ((b & 0x7FFFFFu) > 0x600000u ? 1 : 0);   // 448 = 1.75 x 2^8
  return e < -123 ? -123 : (e > 120 ? 120 : e);
}

template <int N>
__device__ __forceinline__ void vm_wait() { asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory"); }

// Wait until at most n vector-memory operations of this wave are outstanding;
// n is rounded down to an available immediate, which only waits longer.
__device__ __forceinline__ void vm_wait_le(int n) {
  if (n == 8) vm_wait<8>();
  else if (n >= 32) {
    if (n >= 63) vm_wait<63>();
    else if (n >= 48) vm_wait<48>();
    else if (n >= 40) vm_wait<40>();
    else vm_wait<32>();
  } else if (n >= 16) {
    if (n >= 28) vm_wait<28>();
    else if (n >= 24) vm_wait<24>();
    else if (n >= 20) vm_wait<20>();
    else vm_wait<16>();
  } else if (n >= 12) vm_wait<12>();
  else if (n >= 8) vm_wait<8>();
  else if (n >= 4) vm_wait<4>();
  else vm_wait<0>();
}

}  // namespace bf16k

template <int D, bool FP8, bool QK8>
__global__ void __launch_bounds__(512, 1) attn_bf16_kernel(const AttnArgs a, const Plan plan_arg) {
  using namespace bf16k;
  using C = Cfg<D, FP8>;
  static_assert(!QK8 || (FP8 && D == 128), "fp8 scores: E4M3 KV with 128 dims (one 128-deep MFMA per key tile)");
  constexpr int TT = C::kTT;
  constexpr int CPR = C::kCPR;
  constexpr int KS = D / 32;   // k-steps of S^T
  constexpr int DT = D / 16;   // d-tiles of O^T
  __shared__ __attribute__((aligned(1024))) uint8_t lds[C::kLdsBytes];
  __shared__ Plan splan;
#ifdef SPECGEN_TIMELINE
  __shared__ uint64_t tl_t[kTlSlots];
  __shared__ int32_t tl_k[kTlSlots];
#define SG_TL(i, k)                                          \
  do {                                                       \
    if (threadIdx.x == 0) {                                  \
      tl_t[(i)] = __builtin_amdgcn_s_memrealtime();          \
      tl_k[(i)] = (k);                                       \
    }                                                        \
  } while (0)
  // wave 0 writes stamps 0 .. lead - 1 and the end stamp out
  auto tl_flush = [&](int lead) {
    if (threadIdx.x < 64 && blockIdx.x < kTlWorkers) {
      for (int i = threadIdx.x; i < kTlSlots; i += 64) {
        if (i < lead || i == kTlSlots - 1) {
          g_tl_stamp[blockIdx.x][i] = tl_t[i];
          g_tl_kind[blockIdx.x][i] = tl_k[i];
        }
      }
    }
  };
#else
#define SG_TL(i, k) \
  do {              \
  } while (0)
#endif
  SG_TL(0, 100);
  plan_to_lds<512>(plan_arg, splan);
  SG_TL(1, 101);
  const Plan& plan = splan;
  int32_t* items = reinterpret_cast<int32_t*>(lds + C::kOffItems);
  float* ml = reinterpret_cast<float*>(lds + C::kOffML);

  const PartPlan& pp = plan.part[kPartMfma];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = uniform(tid >> 6);
  const int w = blockIdx.x;
  // the walk of the worker's range and the gather of every block id it reads
  // (the ML area is free until the first item ends)
  const WorkerRange wr = worker_walk_tiles<C::kThreads, C::kItemCap, C::kIdsPerTile>(
      a, plan, kPartMfma, w, items, reinterpret_cast<int32_t*>(lds + C::kOffIds), reinterpret_cast<int32_t*>(ml));
  SG_TL(2, 102);
  // The walk reads LDS, so the compiler cannot prove its results uniform;
  // without these readfirstlanes every loop-carried value of the slot loop
  // would live in VGPRs under exec masks.
  const int R = uniform(wr.R);
  const int first_ord = uniform(wr.first_ord);
  const int nitems = uniform(wr.nitems);
  if (R <= 0) {
#ifdef SPECGEN_TIMELINE
    SG_TL(kTlSlots - 1, 0);
    tl_flush(3);
#endif
    return;
  }
  const uint32_t lds_base = (uint32_t)(size_t)((SG_LDS uint8_t*)lds);

  // Item descriptors are read from LDS once per item and kept in scalar registers.
  struct Desc {
    int kind, t, f, j, ord, tile0, ntile, nv, nrows, row0, lastblk, rtile0;
  };
  auto load_desc = [&](int ii) {
    typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
    const SG_LDS i32x4* p = reinterpret_cast<const SG_LDS i32x4*>((SG_LDS uint8_t*)lds + C::kOffItems + ii * kItemInts * 4);
    const i32x4 v0 = p[0], v1 = p[1], v2 = p[2], v3 = p[3];
    static_assert(IT_KIND == 0 && IT_T == 1 && IT_F == 2 && IT_J == 3 && IT_ORD == 5 && IT_TILE0 == 6 &&
                  IT_NTILE == 7 && IT_NVALID == 8 && IT_NROWS == 10 && IT_ROW0 == 11 && IT_RTILE0 == 12 &&
                  IT_LASTBLK == 14, "descriptor layout");
    Desc d;
    d.kind = uniform(v0[0]);
    d.t = uniform(v0[1]);
    d.f = uniform(v0[2]);
    d.j = uniform(v0[3]);
    d.ord = uniform(v1[1]);
    d.tile0 = uniform(v1[2]);
    d.ntile = uniform(v1[3]);
    d.nv = uniform(v2[0]);
    d.nrows = uniform(v2[2]);
    d.row0 = uniform(v2[3]);
    d.lastblk = uniform(v3[2]);
    d.rtile0 = uniform(v3[0]);
    return d;
  };

  // ---- issue side ------------------------------------------------------------
  const int64_t head_stride = (int64_t)D * 2;   // bytes between q heads of a fork
  const int64_t slice_stride = C::kSliceB;      // bytes between kv heads of a block
  const int64_t blk_stride = (int64_t)plan.Hkv * slice_stride;
  const bool is_v = wave >= 4;                  // waves 0-3 move K, waves 4-7 move V
  const int wq = wave & 3;
  // Lane constants for piece i of slice b of this wave (tile block
  // kb = wq * kSlicesPerWave + b).  K: LDS chunk p of tile token row tt holds
  // source chunk p ^ swz_k(tt).  V: the slice is D rows of 32 bytes (16 tokens);
  // lane L of piece i gathers the half that v_pos places at 1024 i + 16 L (a
  // permutation inside the piece's 32 rows).  One instruction moves 1 KiB of
  // the slice.
  constexpr int NB = C::kSlicesPerWave, NI = C::kPiecesPerSlice;
  uint32_t src_off[NB][NI];   // byte offset in the block slice, full tile
  int ptok[NI];               // K: token row of the slice this lane moves
#pragma unroll
  for (int i = 0; i < NI; ++i) ptok[i] = i * C::kRPI + lane / CPR;
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      if (is_v) {
        int d = 0, h = 0;
        v_slot_source(i, lane, wq * NB + b, &d, &h);
        src_off[b][i] = (uint32_t)(32 * d + 16 * h);
      } else {
        const int tt = (wq * NB + b) * 16 + ptok[i];
        src_off[b][i] = (uint32_t)(ptok[i] * C::kRowB + (((lane % CPR) ^ swz_k<CPR>(tt)) << 4));
      }
    }
  // physical id of slice b of this wave in tile k of item d, from the ids the worker gathered into LDS
  const int32_t* ids = reinterpret_cast<const int32_t*>(lds + C::kOffIds);
  auto block_id = [&](const Desc& d, int k, int b) -> int {
    return uniform(ids[(d.rtile0 + k) * C::kIdsPerTile + wq * NB + b]);
  };
  auto issue_slot = [&](const Desc& d, int k, const int (&id)[NB], int stage) {
    const uint32_t st = lds_base + (uint32_t)(stage * C::kStageB);
    if (k < 0) {
      // q rows of the item (rows past its end repeat its last row)
#pragma unroll
      for (int i = 0; i < C::kDmaSlot; ++i) {
        const int n = wave * C::kDmaSlot + i;
        const int row = (n * C::kRPI + lane / CPR) & (C::kQRows - 1);   // row within the slot
        const int rq = row + (q_slots(d.nrows) + k) * C::kQRows;        // row within the item
        const int rr = rq < d.nrows ? rq : d.nrows - 1;
        int fork = 0, hq = 0;
        item_row_fork_head(plan, d.kind, d.t, d.f, d.j, d.row0, rr, &fork, &hq);
        const int chunk = (lane % CPR) ^ swz_q<D>(row);
        const uint32_t voff = (uint32_t)(((int64_t)fork * plan.Hq + hq) * head_stride) + (uint32_t)(chunk * 16);
        dma16_cached(a.q, voff, st + (uint32_t)(n * 1024));
      }
    } else if constexpr (FP8) {
      // this wave's block slices of the tile's K (waves 0-3) or V (waves 4-7)
      // codes, as they are
      constexpr int NI8 = C::kF8Slice / 1024;
      const uint8_t* pool = is_v ? a.v_pool : a.k_pool;
      const int64_t blk8 = (int64_t)plan.Hkv * C::kF8Slice;
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const int kb = wq * NB + b;
        const uint8_t* sb = pool + (int64_t)id[b] * blk8 + (int64_t)d.j * C::kF8Slice;
#pragma unroll
        for (int i = 0; i < NI8; ++i) {
          uint32_t src = (uint32_t)(1024 * i + 16 * lane);
          if (!QK8 && !is_v && D == 128) {
            // K codes of the row and dims this slot's converting lane takes
            src = (uint32_t)(1024 * i + 128 * kdec_row(lane) + 8 * kdec_c0(lane));
          } else if (QK8 && !is_v) {
            // K codes stay codes: 16-byte chunk c of tile row t lands at chunk
            // c ^ k8_swz(t) of its LDS row, so the score reads hit distinct banks
            const int t = 8 * (kb * NI8 + i) + lane / 8;
            src = (uint32_t)(1024 * i + 128 * (lane / 8) + 16 * ((lane % 8) ^ k8_swz(t)));
          }
          dma16(sb, src, st + (uint32_t)((is_v ? C::kTileB : 0) + 2048 * (kb * NI8 + i)));
        }
      }
    } else {
      const int tile = d.tile0 + k;
      const uint8_t* pool = is_v ? a.v_pool : a.k_pool;
      const uint32_t tens = is_v ? (uint32_t)C::kTileB : 0u;
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const int kb = wq * NB + b;   // block within the tile
        const uint8_t* sb = pool + (int64_t)id[b] * blk_stride + d.j * slice_stride;
#pragma unroll
        for (int i = 0; i < NI; ++i) {
          uint32_t off = src_off[b][i];
          if (!is_v && (tile + 1) * TT > d.nv) {
            // K rows of tokens past the item's end re-read its last valid token
            // (finite; their scores are masked).  V slices are moved whole: the
            // math zeroes the values of tokens past the end.
            int bi = tile * C::kIdsPerTile + kb;
            bi = bi < d.lastblk ? bi : d.lastblk;
            int tok = tile * TT + kb * 16 + ptok[i];
            tok = tok < d.nv ? tok : d.nv - 1;
            off = (uint32_t)((tok - bi * 16) * C::kRowB) + (off & (uint32_t)(C::kRowB - 1));
          }
          dma16(sb, off, st + tens + (uint32_t)(kb * C::kSliceB + i * 1024));
        }
      }
    }
  };

  // E4M3: once a tile slot has landed (one iteration before it is computed),
  // every wave turns its K code piece and V code piece (lane: one 16-byte chunk
  // of each) into the bf16 layout the MFMA path reads -- K rows swizzled, V^T
  // halves placed by v_pos -- inside the 2 KiB runs
  // that hold them: it reads its codes before it writes (one wave's LDS
  // operations run in order), and no other wave touches those runs, so no
  // barrier; the next iteration's barrier publishes the tile.  Codes of tokens
  // past an item's end are converted too; their scores and values are masked
  // later, as for bf16.
  auto convert_tile = [&](int stage) {
    uint8_t* st8 = lds + stage * C::kStageB;
    const u32x4 ck = *reinterpret_cast<const u32x4*>(st8 + 2048 * wave + 16 * lane);
    const u32x4 cv = *reinterpret_cast<const u32x4*>(st8 + C::kTileB + 2048 * wave + 16 * lane);
    const int o = tid * 16;   // byte of the chunk within the tile's codes of one tensor
    // K chunk: 16 dims of one token row of block slice kb (fp8 scores read the codes as they are)
    if constexpr (!QK8) {
      const int kb = o / C::kF8Slice;
      const int tok = D == 128 ? 8 * (wave & 1) + kdec_row(lane) : (o % C::kF8Slice) / D;
      const int c8 = D == 128 ? kdec_c0(lane) : (o % D) / 8;   // first bf16 chunk of the 16 dims
      const int tt = kb * 16 + tok;
      const u32x2 b0 = e4m3x4_to_bf16x4(ck[0]), b1 = e4m3x4_to_bf16x4(ck[1]);
      const u32x2 b2 = e4m3x4_to_bf16x4(ck[2]), b3 = e4m3x4_to_bf16x4(ck[3]);
      const int sw = swz_k<CPR>(tt);
      *reinterpret_cast<u32x4*>(st8 + tt * C::kRowB + ((c8 ^ sw) << 4)) = u32x4{b0[0], b0[1], b1[0], b1[1]};
      *reinterpret_cast<u32x4*>(st8 + tt * C::kRowB + (((c8 + 1) ^ sw) << 4)) = u32x4{b2[0], b2[1], b3[0], b3[1]};
    }
    // V chunk: the 16 tokens of row d of block slice kb
    {
      const int kb = o / C::kF8Slice;
      const int dd = (o % C::kF8Slice) / 16;
      uint8_t* vs = st8 + C::kTileB + kb * C::kSliceB;
      const u32x2 b0 = e4m3x4_to_bf16x4(cv[0]), b1 = e4m3x4_to_bf16x4(cv[1]);
      const u32x2 b2 = e4m3x4_to_bf16x4(cv[2]), b3 = e4m3x4_to_bf16x4(cv[3]);
      *reinterpret_cast<u32x4*>(vs + v_pos(dd, 0, kb)) = u32x4{b0[0], b0[1], b1[0], b1[1]};
      *reinterpret_cast<u32x4*>(vs + v_pos(dd, 1, kb)) = u32x4{b2[0], b2[1], b3[0], b3[1]};
    }
  };
  static_assert(!FP8 || C::kTT * D == 16 * C::kThreads, "one K and one V code chunk per thread");
  static_assert(!FP8 || 2 * C::kTileB == 2048 * 2 * C::kWaves, "a 2 KiB run of each tensor per wave");

  // ---- compute side ------------------------------------------------------------
  const int G = lane >> 4;     // 16-lane group
  const int ln = lane & 15;    // row within an N-tile / key within an S^T tile
  const int k_lane_tok = 8 * (ln >> 2) + (ln & 3);
  const int k_lane_swz = swz_k<CPR>(k_lane_tok);
  // V^T operand of d-tile dt for a slab at token sb: block sb/16 + G/2 of the
  // tile (sb/16 is even, so the block's parity is that of G/2), row d = 16 dt +
  // ln, half G & 1, at v_pos(ln, G & 1, G / 2) + 512 dt of the slice
  static_assert(TT % 32 == 0, "slabs start at even blocks");
  const int v_lane_off = (G >> 1) * C::kSliceB + v_pos(ln, G & 1, G >> 1);
  bf16x8 qop[2][KS];
  // QK8: per N-tile, the E4M3 codes of the lane's 32 dims of its row (dims
  // 16G .. 16G+15 in bytes 0-15, 64+16G .. +15 in bytes 16-31, the operand
  // layout of the 128-deep fp8 MFMA) for both terms, and their E8M0 scales
  i32x8 q8h[2], q8l[2];
  int q8sh[2], q8sl[2];
  f32x4 acc[2][DT];
  // Per row (each lane: its share of it): the running max, and two sums of
  // the probabilities: l_run of the bf16 weights the PV product uses (the
  // output's normaliser, so a dominant key's rounding cancels out of the
  // output) and lf_run of the unrounded fp32 ones (the lse, which would
  // otherwise carry that rounding, up to 2^-8 relative).
  float m_run[2], l_run[2], lf_run[2];
  constexpr int NT = 2;   // 16-row MFMA tiles per row group
  int RG = 1, TG = 1, rg = 0, tg = 0, tpg = TT;   // tpg: tokens of a tile per token group
  bool active = false;

  // q slot qi (of 1 or 2) of an item: sets up the item's wave layout and
  // clears the accumulators (again at the second q slot, where no tile of the
  // item has run yet), and the waves whose 32 rows are in this slot read their
  // Q^T operands from it.
  auto begin_item = [&](const Desc& d, int stage, int qi) {
    const int nrows = d.nrows;
    constexpr int RS = 16 * NT;
    RG = (nrows + RS - 1) / RS;
    TG = (TT / 32) < (C::kWaves / RG) ? (TT / 32) : (C::kWaves / RG);
    rg = wave % RG;
    tg = wave / RG;
    tpg = TT / TG;
    active = wave < RG * TG;
    const SG_LDS uint8_t* qb = (const SG_LDS uint8_t*)lds + stage * C::kStageB;
    const bool mine = (rg * RS) / C::kQRows == qi;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int row = rg * RS + nt * 16 + ln - qi * C::kQRows;   // row within the slot
      if (QK8 && mine) {
        // the row's largest |q| over its 4 lanes (the 4 lane groups hold a
        // quarter of its dims each) sets e; every lane computes it (`mine` is
        // wave-uniform: only the waves whose rows are in this slot read it)
        const SG_LDS uint8_t* qr = qb + row * C::kRowB;
        u32x4 c4[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int ch = (i < 2 ? 2 * G + i : 8 + 2 * G + (i - 2)) ^ swz_q<D>(row);
          c4[i] = *reinterpret_cast<const SG_LDS u32x4*>(qr + ch * 16);
        }
        float x[32];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const uint32_t w0 = c4[i].x, w1 = c4[i].y, w2 = c4[i].z, w3 = c4[i].w;
          const uint32_t ww[4] = {w0, w1, w2, w3};
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            x[8 * i + 2 * j] = __uint_as_float(ww[j] << 16);
            x[8 * i + 2 * j + 1] = __uint_as_float(ww[j] & 0xFFFF0000u);
          }
        }
        float amax = 0.f;
#pragma unroll
        for (int i = 0; i < 32; ++i) amax = fmaxf(amax, fabsf(x[i]));
        amax = rows4_max(amax);
        const int e = q8_exponent(amax);
        const float inv = __uint_as_float((uint32_t)(127 - e) << 23);   // 2^-e, exact
        uint32_t hw[8], lw[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          // four values: codes of x * 2^-e (RNE), then of the remainder times 16
          const float y0 = x[4 * k] * inv, y1 = x[4 * k + 1] * inv, y2 = x[4 * k + 2] * inv, y3 = x[4 * k + 3] * inv;
          uint32_t h = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(y0, y1, 0, false);
          h = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(y2, y3, (int)h, true);
          const f32x2 d01 = __builtin_amdgcn_cvt_pk_f32_fp8((int)h, false);
          const f32x2 d23 = __builtin_amdgcn_cvt_pk_f32_fp8((int)h, true);
          uint32_t l = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32((y0 - d01[0]) * 16.f, (y1 - d01[1]) * 16.f, 0, false);
          l = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32((y2 - d23[0]) * 16.f, (y3 - d23[1]) * 16.f, (int)l, true);
          hw[k] = h;
          lw[k] = l;
        }
        q8h[nt] = i32x8{(int)hw[0], (int)hw[1], (int)hw[2], (int)hw[3], (int)hw[4], (int)hw[5], (int)hw[6], (int)hw[7]};
        q8l[nt] = i32x8{(int)lw[0], (int)lw[1], (int)lw[2], (int)lw[3], (int)lw[4], (int)lw[5], (int)lw[6], (int)lw[7]};
        q8sh[nt] = 127 + e;
        q8sl[nt] = 127 + e - 4;
      } else if (!QK8 && mine) {
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const int slot = (ks * 4 + G) ^ swz_q<D>(row);
          qop[nt][ks] = *reinterpret_cast<const SG_LDS bf16x8*>(qb + row * C::kRowB + slot * 16);
        }
      }
      m_run[nt] = -INFINITY;
      l_run[nt] = 0.f;
      lf_run[nt] = 0.f;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) acc[nt][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
  };


  // one 32-token slab starting at token sb of the tile in `stage`; `valid` tokens of the tile are real
  auto slab = [&](auto mask_c, int stage, int sb, int valid, int idb) {
    constexpr bool kMask = decltype(mask_c)::value;   // the slab runs past the tile's valid tokens
    const SG_LDS uint8_t* kb = (const SG_LDS uint8_t*)lds + stage * C::kStageB;
    const SG_LDS uint8_t* vb = kb + C::kTileB;
    // V^T operands: lane (G, ln) reads V[sb+8G+0..7][16dt+ln] in one 16-byte
    // load.  They are read with the keys, so the reads overlap the score MFMAs
    // and the softmax rather than waiting in front of the PV product.
    u32x4 vkeep = {~0u, ~0u, ~0u, ~0u};   // masked slab: keep only the values of valid tokens
    if constexpr (kMask) {
#pragma unroll
      for (int e2 = 0; e2 < 4; ++e2) {
        const int t0 = sb + 8 * G + 2 * e2;
        vkeep[e2] = (t0 < valid ? 0x0000FFFFu : 0u) | (t0 + 1 < valid ? 0xFFFF0000u : 0u);
      }
    }
    f32x4 s[2][NT];
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) s[u][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
    const SG_LDS uint8_t* vrow = vb + (sb >> 4) * C::kSliceB + v_lane_off;
    u32x4 vraw[DT];
    if constexpr (QK8) {
      // A operand: key row t's codes, dims 16G .. +15 and 64+16G .. +15 (chunks G
      // and 4+G, swizzled), for the keys {8G' + e} (u = 0) and {8G' + 4 + e} (u = 1)
      i32x8 k8[2];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int t = sb + k_lane_tok + 4 * u;
        const SG_LDS uint8_t* krow = kb + (t >> 3) * 2048 + (t & 7) * 128;
        const int sw = k8_swz(t);
        const u32x4 lo = *reinterpret_cast<const SG_LDS u32x4*>(krow + ((G ^ sw) << 4));
        const u32x4 hi = *reinterpret_cast<const SG_LDS u32x4*>(krow + (((4 + G) ^ sw) << 4));
        k8[u] = i32x8{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
      }
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) vraw[dt] = *reinterpret_cast<const SG_LDS u32x4*>(vrow + dt * 512);
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          s[u][nt] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(k8[u], q8l[nt], s[u][nt], 0, 0, 0, 127, 0,
                                                                       q8sl[nt]);
          s[u][nt] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(k8[u], q8h[nt], s[u][nt], 0, 0, 0, 127, 0,
                                                                       q8sh[nt]);
        }
    } else {
      const SG_LDS uint8_t* ka_row = kb + (sb + k_lane_tok) * C::kRowB;
      const SG_LDS uint8_t* kb_row = ka_row + 4 * C::kRowB;
      bf16x8 ka[KS], kbo[KS];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const int cho = (((4 * ks + G) ^ k_lane_swz) << 4);
        ka[ks] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const SG_LDS u32x4*>(ka_row + cho));
        kbo[ks] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const SG_LDS u32x4*>(kb_row + cho));
      }
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) vraw[dt] = *reinterpret_cast<const SG_LDS u32x4*>(vrow + dt * 512);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          s[0][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka[ks], qop[nt][ks], s[0][nt], 0, 0, 0);
          s[1][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kbo[ks], qop[nt][ks], s[1][nt], 0, 0, 0);
        }
      }
    }
    // lane (G, ln) holds, for row ln of each N-tile, the scores of keys sb+8G+0..7
    // (all in block (sb + 8G) / 16 of the tile)
    // E4M3: the key scale multiplies a slab's scores only where the slab is
    // masked; elsewhere it rides in the exponent's scale factor, cl, and in the
    // row maxima (scales are non-negative, so scaling commutes with max).  The
    // value scale rides in the exponent's offset (log2 vsc): the exponentials
    // give P times the value scale, which the PV product takes as it is.
    float inv_vsc = 1.f, lvs = 0.f, ksc = 1.f;
    if constexpr (FP8) {
      // the slab's two blocks (ids[idb + sb/16] and the next): lanes G < 2 hold
      // keys of the first, lanes G >= 2 keys of the second.  Scalar loads (the
      // constant address space): a vector load would sit in the vmcnt queue
      // behind the slots in flight.
      typedef const __attribute__((address_space(4))) float* cfp;
      const int id0 = uniform(ids[idb + (sb >> 4)]);
      const int id1 = uniform(ids[idb + (sb >> 4) + 1]);
      const cfp ks = (cfp)a.k_scale;
      const cfp vs = (cfp)a.v_scale;
      // (each value is pinned wave-uniform, so the two loads are not merged
      // into one per-lane load of a selected address)
      auto sload = [](cfp p, int i) { return __int_as_float(uniform(__float_as_int(p[i]))); };
      const float k0 = sload(ks, id0), k1 = sload(ks, id1), v0 = sload(vs, id0), v1 = sload(vs, id1);
      ksc = G < 2 ? k0 : k1;
      // A block whose value scale is 0 holds zero values: its lanes zero their
      // V operands and take scale 1 for P, so its keys still count in the sums.
      if (v0 == 0.f || v1 == 0.f) {
        const bool zv = (G < 2 ? v0 : v1) == 0.f;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
          if (zv) vraw[dt] = u32x4{0u, 0u, 0u, 0u};
      }
      const float ve = G < 2 ? v0 : v1;
      const float vsc = ve > 0.f ? ve : 1.f;
      inv_vsc = __builtin_amdgcn_rcpf(vsc);
      lvs = __builtin_amdgcn_logf(vsc);
      if constexpr (kMask) {   // scaled before the -inf masking (a zero scale times -inf would be NaN)
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
          for (int nt = 0; nt < NT; ++nt) s[u][nt] *= ksc;
        ksc = 1.f;
      }
    }
    if constexpr (kMask) {
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (sb + 8 * G + 4 * u + e >= valid) {
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) s[u][nt][e] = -INFINITY;
          }
    }
    // this lane's max over its 8 scores of each row; the row max (over the 4
    // lanes of a row) is only needed when the reference max moves
    float mx[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
      mx[nt] = ksc * fmaxf(fmaxf(fmaxf(s[0][nt][0], s[0][nt][1]), fmaxf(s[0][nt][2], s[0][nt][3])),
                           fmaxf(fmaxf(s[1][nt][0], s[1][nt][1]), fmaxf(s[1][nt][2], s[1][nt][3])));
    // Lazy rescaling: the reference max only moves when a score exceeds it by
    // more than 2^kRescaleLog2 in probability (one wave-uniform decision for
    // both N-tiles; m_run is the same on the 4 lanes of a row).
    if (__builtin_amdgcn_ballot_w64(mx[0] * a.c_log2 > m_run[0] * a.c_log2 + kRescaleLog2 ||
                                   mx[1] * a.c_log2 > m_run[1] * a.c_log2 + kRescaleLog2)) {
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const float m_new = fmaxf(m_run[nt], rows4_max(mx[nt]));
        const float alpha = __builtin_amdgcn_exp2f((m_run[nt] - m_new) * a.c_log2);
        m_run[nt] = m_new;
        l_run[nt] *= alpha;
        lf_run[nt] *= alpha;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) acc[nt][dt] *= alpha;
      }
    }
    bf16x8 vop[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      u32x4 vv = vraw[dt];
      if constexpr (kMask) vv &= vkeep;   // values past the end may be any bits, NaN included
      vop[dt] = __builtin_bit_cast(bf16x8, vv);
    }
    // P = exp2(S - m) in bf16, then O^T += V^T P^T; the exponentials of N-tile 1
    // are interleaved with the PV MFMAs of N-tile 0
    const float mc0 = m_run[0] * a.c_log2 - lvs, mc1 = m_run[1] * a.c_log2 - lvs;
    const float cl = a.c_log2 * ksc;
    float p0[8], p1[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      p0[e] = __builtin_amdgcn_exp2f(fmaf(s[0][0][e], cl, -mc0));
      p0[4 + e] = __builtin_amdgcn_exp2f(fmaf(s[1][0][e], cl, -mc0));
    }
    // the sums take P without the value scale
    const float sp0 = ((p0[0] + p0[1]) + (p0[2] + p0[3])) + ((p0[4] + p0[5]) + (p0[6] + p0[7]));
    if constexpr (FP8) lf_run[0] = fmaf(sp0, inv_vsc, lf_run[0]);
    else lf_run[0] += sp0;
    u32x4 pk0;
    pk0[0] = pack_bf16x2(p0[0], p0[1]);
    pk0[1] = pack_bf16x2(p0[2], p0[3]);
    pk0[2] = pack_bf16x2(p0[4], p0[5]);
    pk0[3] = pack_bf16x2(p0[6], p0[7]);
    // the normaliser adds the weights PV uses, without the value scale
    if constexpr (FP8) l_run[0] = fmaf(row_sum_bf16(pk0, 0.f), inv_vsc, l_run[0]);
    else l_run[0] = row_sum_bf16(pk0, l_run[0]);
    const bf16x8 pop0 = __builtin_bit_cast(bf16x8, pk0);
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      acc[0][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vop[dt], pop0, acc[0][dt], 0, 0, 0);
      if (dt < 8) p1[dt] = __builtin_amdgcn_exp2f(fmaf(s[dt >> 2][1][dt & 3], cl, -mc1));
    }
#pragma unroll
    for (int e = DT; e < 8; ++e)   // D = 64: fewer PV MFMAs than exponentials
      p1[e] = __builtin_amdgcn_exp2f(fmaf(s[e >> 2][1][e & 3], cl, -mc1));
    const float sp1 = ((p1[0] + p1[1]) + (p1[2] + p1[3])) + ((p1[4] + p1[5]) + (p1[6] + p1[7]));
    if constexpr (FP8) lf_run[1] = fmaf(sp1, inv_vsc, lf_run[1]);
    else lf_run[1] += sp1;
    u32x4 pk1;
    pk1[0] = pack_bf16x2(p1[0], p1[1]);
    pk1[1] = pack_bf16x2(p1[2], p1[3]);
    pk1[2] = pack_bf16x2(p1[4], p1[5]);
    pk1[3] = pack_bf16x2(p1[6], p1[7]);
    if constexpr (FP8) l_run[1] = fmaf(row_sum_bf16(pk1, 0.f), inv_vsc, l_run[1]);
    else l_run[1] = row_sum_bf16(pk1, l_run[1]);
    const bf16x8 pop1 = __builtin_bit_cast(bf16x8, pk1);
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) acc[1][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vop[dt], pop1, acc[1][dt], 0, 0, 0);
    // pin the interleave: (MFMA, TRANS, VALU) x 8 after N-tile 0's softmax
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x400, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x002, 1, 0);
    }
  };

  auto compute_tile = [&](const Desc& d, int k, int stage) {
    if (!active) return;
    const int tile = d.tile0 + k;
    const int rem = d.nv - tile * TT;
    const int valid = rem < TT ? rem : TT;
    const int tok0 = tg * tpg;
    const int tok1 = (tok0 + tpg) < valid ? (tok0 + tpg) : valid;   // this wave's tokens: [tok0, tok1)
    const int idb = (d.rtile0 + k) * C::kIdsPerTile;   // the tile's block ids in LDS
    int sb = tok0;
    for (; sb + 32 <= tok1; sb += 32) slab(std::integral_constant<bool, false>(), stage, sb, valid, idb);
    if (sb < tok1) slab(std::integral_constant<bool, true>(), stage, sb, valid, idb);   // partial last slab
  };

  // Combine the token groups of the item through the stage just consumed and
  // write the normalised partial (o, lse) of each row.  Every wave calls this
  // (it has barriers); returns the number of vector-memory stores this wave
  // issued.
  //   Two token groups (every D = 128 item of up to 128 rows): the waves of a
  // row-group pair swap halves -- token group 0 keeps N-tile 0 and sends
  // N-tile 1, token group 1 the reverse -- so each wave combines and stores
  // one N-tile.  The sent half travels normalised by its row sum, as fp16
  // with the per-row power-of-two scale of the stored partials (4 KiB per
  // wave: 32 KiB, one stage, for eight waves), and its (m, l, lf, scale)
  // through the ML area.
  //   More token groups (D = 64): token group 0 gathers the others' fp32
  // accumulators in rounds that fit the stage and stores both N-tiles.
  auto finish_item = [&](const Desc& d, int stage) -> int {
    float lrow[2], lfrow[2];
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
      lrow[nt] = rows4_sum(l_run[nt]);
      lfrow[nt] = rows4_sum(lf_run[nt]);
    }
    int nt_lo = 0;   // this wave stores N-tiles nt_lo .. NT - 1 (TG = 2: only nt_lo)
    bool stores = active && tg == 0;
    // (keep is a compile-time constant in each call, so the accumulator arrays
    // are indexed statically and stay in registers)
    auto swap_halves = [&](auto keep_c) {
      constexpr int keep = decltype(keep_c)::value, send = 1 - keep;
      uint32_t* cb = reinterpret_cast<uint32_t*>(lds + stage * C::kStageB);
      lds_barrier();   // every wave is done with the stage's K and V
      if (active) {
        const float inv_l = lrow[send] > 0.f ? 1.f / lrow[send] : 0.f;
        float amax = 0.f;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
          for (int e = 0; e < 4; ++e) amax = fmaxf(amax, fabsf(acc[send][dt][e]));
        amax = rows4_max(amax);
        const uint32_t kexp = (uint32_t)part_row_k(__float_as_uint(amax * inv_l));
        const float mul = inv_l * __uint_as_float((254u - kexp) << 23);
        // chunk c (d-tiles 2c, 2c + 1) of lane L at 1 KiB * c + 16 B * L of the wave's region
#pragma unroll
        for (int c = 0; c < DT / 2; ++c) {
          const f32x4 x = acc[send][2 * c] * mul, y = acc[send][2 * c + 1] * mul;
          const u32x4 ch = {pack_f16x2(x[0], x[1]), pack_f16x2(x[2], x[3]), pack_f16x2(y[0], y[1]),
                            pack_f16x2(y[2], y[3])};
          *reinterpret_cast<u32x4*>(cb + (wave * (DT / 2) + c) * 256 + lane * 4) = ch;
        }
        if (G == 0)
          *reinterpret_cast<f32x4*>(ml + ((wave * 2 + send) * 16 + ln) * 4) =
              f32x4{m_run[send], lrow[send], lfrow[send], __uint_as_float(kexp << 23)};
      }
      lds_barrier();
      if (active) {
        const int pw = rg + (1 - tg) * RG;   // the partner wave (same row group)
        const f32x4 ml1 = *reinterpret_cast<const f32x4*>(ml + ((pw * 2 + keep) * 16 + ln) * 4);
        const float m1 = ml1[0], l1 = ml1[1], lf1 = ml1[2];
        // a token group that saw no token of the item has m = -inf, l = 0 and sent zeros
        const float m = fmaxf(m_run[keep], m1);
        const float mc = (m == -INFINITY) ? 0.f : m * a.c_log2;
        const float a0 = __builtin_amdgcn_exp2f(m_run[keep] * a.c_log2 - mc);
        const float a1 = __builtin_amdgcn_exp2f(m1 * a.c_log2 - mc);
        const float w1 = a1 * l1 * ml1[3];   // the partner's accumulator is o1 * l1 * scale
#pragma unroll
        for (int c = 0; c < DT / 2; ++c) {
          const u32x4 ch = *reinterpret_cast<const u32x4*>(cb + (pw * (DT / 2) + c) * 256 + lane * 4);
          const f32x2 x01 = unpack_f16x2(ch[0]), x23 = unpack_f16x2(ch[1]);
          const f32x2 y01 = unpack_f16x2(ch[2]), y23 = unpack_f16x2(ch[3]);
          acc[keep][2 * c] = acc[keep][2 * c] * a0 + f32x4{x01[0], x01[1], x23[0], x23[1]} * w1;
          acc[keep][2 * c + 1] = acc[keep][2 * c + 1] * a0 + f32x4{y01[0], y01[1], y23[0], y23[1]} * w1;
        }
        lrow[keep] = lrow[keep] * a0 + l1 * a1;
        lfrow[keep] = lfrow[keep] * a0 + lf1 * a1;
        m_run[keep] = m;
      }
    };
    if (TG == 2) {
      if (tg == 0) swap_halves(std::integral_constant<int, 0>());
      else swap_halves(std::integral_constant<int, 1>());
      nt_lo = tg;
      stores = active;
    } else if (TG > 2) {
      float* cb = reinterpret_cast<float*>(lds + stage * C::kStageB);
      constexpr int wave_bytes = NT * DT * 64 * 16;
      const int per_round = C::kStageB / wave_bytes;      // writers whose accumulators fit at once
      const int writers = (TG - 1) * RG;
      const int rounds = (writers + per_round - 1) / per_round;
      const int windex = (tg - 1) * RG + rg;              // this wave as a writer (tg >= 1)
      for (int r = 0; r < rounds; ++r) {
        lds_barrier();
        if (active && tg >= 1 && windex / per_round == r) {
          float* dst = cb + (windex % per_round) * (wave_bytes / 4);
#pragma unroll
          for (int nt = 0; nt < NT; ++nt) {
#pragma unroll
            for (int dt = 0; dt < DT; ++dt)
              *reinterpret_cast<f32x4*>(dst + ((nt * DT + dt) * 64 + lane) * 4) = acc[nt][dt];
            // a row's m and sums are the same on its four lanes: lane group 0 writes them
            if (G == 0)
              *reinterpret_cast<f32x4*>(ml + ((wave * 2 + nt) * 16 + ln) * 4) = f32x4{m_run[nt], lrow[nt], lfrow[nt], 0.f};
          }
        }
        lds_barrier();
        if (active && tg == 0) {
          for (int t2 = 1; t2 < TG; ++t2) {
            const int wi = (t2 - 1) * RG + rg;
            if (wi / per_round != r) continue;
            const int pw = t2 * RG + rg;   // the partner wave
            const float* src = cb + (wi % per_round) * (wave_bytes / 4);
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
              // a token group that saw no token of the item has m = -inf, l = 0, acc = 0
              const f32x4 ml1 = *reinterpret_cast<const f32x4*>(ml + ((pw * 2 + nt) * 16 + ln) * 4);
              const float m1 = ml1[0], l1 = ml1[1], lf1 = ml1[2];
              const float m = fmaxf(m_run[nt], m1);
              const float mc = (m == -INFINITY) ? 0.f : m * a.c_log2;
              const float a0 = __builtin_amdgcn_exp2f(m_run[nt] * a.c_log2 - mc);
              const float a1 = __builtin_amdgcn_exp2f(m1 * a.c_log2 - mc);
#pragma unroll
              for (int dt = 0; dt < DT; ++dt) {
                const f32x4 o1 = *reinterpret_cast<const f32x4*>(src + ((nt * DT + dt) * 64 + lane) * 4);
                acc[nt][dt] = acc[nt][dt] * a0 + o1 * a1;
              }
              lrow[nt] = lrow[nt] * a0 + l1 * a1;
              lfrow[nt] = lfrow[nt] * a0 + lf1 * a1;
              m_run[nt] = m;
            }
          }
        }
      }
    }
    if (!stores) return 0;
    const int kseg = d.ord - first_ord;
    const int64_t slot = slot_of(pp, w, kseg);
    if (slot < 0) return 0;
    constexpr int RS = 16 * NT;
    int nst = 0;
    // every lane of an N-tile that holds rows of the item stores (rows past the
    // item's end land in unused rows of the slot), so the count is wave-uniform
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      if (nt < nt_lo || (TG == 2 && nt > nt_lo)) continue;
      if (rg * RS + nt * 16 >= d.nrows) break;
      const int row = rg * RS + nt * 16 + ln;
      // the row's largest |o| (its 4 lanes hold 32 dims each) sets its fp16 scale
      float amax = 0.f;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int e = 0; e < 4; ++e) amax = fmaxf(amax, fabsf(acc[nt][dt][e]));
      amax = rows4_max(amax);
      const float inv_l = 1.f / lrow[nt];
      const uint32_t kexp = (uint32_t)part_row_k(__float_as_uint(amax * inv_l));
      const float mul = inv_l * __uint_as_float((254u - kexp) << 23);
      const float dec = __uint_as_float(kexp << 23);
      uint32_t* orow = reinterpret_cast<uint32_t*>(a.ws + part_o_off(pp, slot, row, D));
      // d-tiles 2p and 2p+1: lane (G, ln) holds dims 16*dt + 4G .. +3 of each;
      // one row swap between lane groups G and G^1 leaves every lane 8
      // consecutive dims, 16*(2p + (G&1)) + 8*(G>>1) .. +7, stored as 16 bytes
      // (the four lanes of a row write 64 contiguous bytes per instruction)
#pragma unroll
      for (int p2 = 0; p2 < DT / 2; ++p2) {
        const f32x4 x = acc[nt][2 * p2] * mul, y = acc[nt][2 * p2 + 1] * mul;
        const auto r0 = __builtin_amdgcn_permlane16_swap(pack_f16x2(x[0], x[1]), pack_f16x2(y[0], y[1]), false, false);
        const auto r1 = __builtin_amdgcn_permlane16_swap(pack_f16x2(x[2], x[3]), pack_f16x2(y[2], y[3]), false, false);
        const u32x4 chunk = {r0[0], r1[0], r0[1], r1[1]};
        const int dim0 = (2 * p2 + (G & 1)) * 16 + 8 * (G >> 1);
        // partials are read once, by the merge: nontemporal stores keep them out
        // of the caches' retention
        __builtin_nontemporal_store(chunk, reinterpret_cast<u32x4*>(orow + dim0 / 2));
      }
      const f32x2 ld = {m_run[nt] * a.sm_scale + __logf(lfrow[nt]), dec};
      __builtin_nontemporal_store(ld, reinterpret_cast<f32x2*>(a.ws + part_l_off(pp, slot, row)));
      nst += DT / 2 + 1;
    }
    return nst;
  };

  // ---- the slot loop -------------------------------------------------------------
  // Slot k of an item: k < 0 its q slots (-q_slots .. -1), then its tiles.
  auto advance = [&](int& ii, int& k, Desc& d) {
    if (k + 1 < d.ntile) {
      ++k;
    } else {
      ++ii;
      if (ii < nitems) {
        d = load_desc(ii);
        k = -q_slots(d.nrows);
      }
    }
  };
  Desc is_d = load_desc(0);
  int S = R;   // slots: each item's q slots, then its tiles
  for (int ii = 0; ii < nitems; ++ii) S += q_slots(uniform(items[ii * kItemInts + IT_NROWS]));
  S = uniform(S);
  int is_ii = 0, is_k = -q_slots(is_d.nrows), issued = 0;   // next slot to issue
  int is_id[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) is_id[b] = 0;
  // Vector-memory operations this wave has issued (DMA instructions and
  // partial stores), and the count right after the DMAs of slots s .. s + 3 of
  // iteration s (the slot issued during iteration s is s + 3): vmcnt retires
  // in order, so slot t has landed once at most ops - mark(t) operations are
  // outstanding.  Fixed roles shifted once per iteration, never an indexed
  // array (which the compiler would place in scratch memory).
  int ops = 0;
  int mk0 = 0, mk1 = 0, mk2 = 0, mk3 = 0;
  auto load_ids = [&]() {   // block ids of the next slot to issue, if it is a tile
    if (issued < S && is_k >= 0) {
#pragma unroll
      for (int b = 0; b < NB; ++b) is_id[b] = block_id(is_d, is_k, b);
    }
  };
  auto issue_next = [&]() {   // slot `issued` into its stage (the one consumed last iteration)
    issue_slot(is_d, is_k, is_id, issued & 3);
    ops += is_k < 0 ? C::kDmaSlot : C::kTileDma;
    advance(is_ii, is_k, is_d);
    ++issued;
    load_ids();   // for the next issue
    return ops;
  };
  // slots 0 .. 2 (slot 0 is the first item's q rows)
  static_assert(C::kStages == 4, "three slots ahead");
  if (issued < S) mk0 = issue_next();
  if (issued < S) mk1 = issue_next();
  if (issued < S) mk2 = issue_next();
  SG_TL(3, 103);
  Desc cp_d = load_desc(0);
  int cp_ii = 0, cp_k = -q_slots(cp_d.nrows);
  // bf16 KV: waves 0-3 queue their share of the next slot's DMAs after their
  // compute, waves 4-7 before it.  Issuing a slot's 32 DMA instructions stalls
  // the issuing waves for hundreds of cycles; with all eight issuing at once
  // after the barrier, the two waves of each SIMD (w and w + 4) then run every
  // phase of the slab (score MFMAs, softmax, PV MFMAs) in step and contend for
  // the same unit.  Staggered, one wave's matrix work overlaps the other's
  // vector work: 1.32 instead of 1.52 us per 32 KiB prefix slot on the 32k-prefix
  // workload.  (E4M3 KV keeps the single issue point: there every wave
  // converts the next tile right after the barrier, and the split gained 2%.)
  const bool late_dma = !FP8 && wave < 4;
  for (int s = 0; s < S; ++s) {
    // E4M3 converts the next tile during this iteration, so it waits for that slot
    vm_wait_le(uniform(ops - ((FP8 && s + 1 < S) ? mk1 : mk0)));
    lds_barrier();
#ifdef SPECGEN_TIMELINE
    if (s < kTlSlots - 5) SG_TL(4 + s, cp_k < 0 ? -1 : cp_d.kind);
#endif
    if (!late_dma && issued < S) mk3 = issue_next();
    const int stage = s & 3;
    if constexpr (FP8) {
      if (s + 1 < S && cp_k + 1 >= 0 && cp_k + 1 < cp_d.ntile) convert_tile((s + 1) & 3);   // slot s + 1 is a tile
    }
    int st0 = 0;
    if (cp_k < 0) {
      begin_item(cp_d, stage, q_slots(cp_d.nrows) + cp_k);
    } else {
      compute_tile(cp_d, cp_k, stage);
      if (cp_k == cp_d.ntile - 1) st0 = uniform(finish_item(cp_d, stage));
    }
    ops += st0;
    // the slot goes into the stage consumed last iteration, which no wave reads
    // again before it lands: late issue only shortens its lead
    if (late_dma && issued < S) mk3 = issue_next();
    mk0 = mk1;
    mk1 = mk2;
    mk2 = mk3;
    advance(cp_ii, cp_k, cp_d);
  }
#ifdef SPECGEN_TIMELINE
  SG_TL(kTlSlots - 1, S);
  tl_flush(4 + (S < kTlSlots - 5 ? S : kTlSlots - 5));
#endif
#undef SG_TL
}

// Partial kernel of the MFMA partition: bf16 KV, or E4M3 KV decoded exactly to
// bf16 in LDS, or (qk8, D = 128 only) E4M3 KV with fp8 scores.
hipError_t launch_attn_mfma_any(const AttnArgs& a, const Plan& plan, bool fp8, bool qk8, hipStream_t stream) {
  const int W = plan.part[kPartMfma].workers;
  if (W <= 0) return hipSuccess;
  if (qk8 && (!fp8 || plan.D != 128)) return hipErrorInvalidValue;
  if (plan.D == 128) {
    if (qk8) hipLaunchKernelGGL((attn_bf16_kernel<128, true, true>), dim3(W), dim3(512), 0, stream, a, plan);
    else if (fp8) hipLaunchKernelGGL((attn_bf16_kernel<128, true, false>), dim3(W), dim3(512), 0, stream, a, plan);
    else hipLaunchKernelGGL((attn_bf16_kernel<128, false, false>), dim3(W), dim3(512), 0, stream, a, plan);
  } else {
    if (fp8) hipLaunchKernelGGL((attn_bf16_kernel<64, true, false>), dim3(W), dim3(512), 0, stream, a, plan);
    else hipLaunchKernelGGL((attn_bf16_kernel<64, false, false>), dim3(W), dim3(512), 0, stream, a, plan);
  }
  return hipGetLastError();
}

int mfma_tile_tokens(int D, bool fp8) {
  (void)fp8;
  return D == 128 ? bf16k::Cfg<128, false>::kTT : bf16k::Cfg<64, false>::kTT;
}
int mfma_tile_cap(int D, bool fp8) {
  (void)fp8;
  return D == 128 ? bf16k::Cfg<128, false>::kTileCap : bf16k::Cfg<64, false>::kTileCap;
}
int mfma_item_cap() { return bf16k::Cfg<128, false>::kItemCap; }
int mfma_walk_threads() { return bf16k::Cfg<128, false>::kThreads; }
int mfma_rows() { return bf16k::Cfg<128, false>::kMaxRows; }

}  // namespace specgen

#ifdef SPECGEN_TIMELINE
// The stamps of the last partial-kernel launches on the current device
// (include/specgen_timeline.h).
extern "C" int specgen_timeline_shape(int* workers, int* slots) {
  if (!workers || !slots) return 1;
  *workers = specgen::kTlWorkers;
  *slots = specgen::kTlSlots;
  return 0;
}
extern "C" int specgen_timeline_read(uint64_t* stamps, int32_t* kinds) {
  if (!stamps || !kinds) return 1;
  if (hipMemcpyFromSymbol(stamps, HIP_SYMBOL(specgen::g_tl_stamp), sizeof(specgen::g_tl_stamp)) != hipSuccess)
    return 2;
  if (hipMemcpyFromSymbol(kinds, HIP_SYMBOL(specgen::g_tl_kind), sizeof(specgen::g_tl_kind)) != hipSuccess) return 2;
  return 0;
}
extern "C" int specgen_timeline_clear(void) {
  void* p = nullptr;
  if (hipGetSymbolAddress(&p, HIP_SYMBOL(specgen::g_tl_stamp)) != hipSuccess ||
      hipMemset(p, 0, sizeof(specgen::g_tl_stamp)) != hipSuccess)
    return 2;
  if (hipGetSymbolAddress(&p, HIP_SYMBOL(specgen::g_tl_kind)) != hipSuccess ||
      hipMemset(p, 0, sizeof(specgen::g_tl_kind)) != hipSuccess)
    return 2;
  return hipDeviceSynchronize() == hipSuccess ? 0 : 2;
}
#endif
