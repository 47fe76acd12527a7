// lds_layout.h -- where the bf16 partial kernel puts K and V^T bytes in LDS,
// and which global bytes each lane's DMA gathers to put them there.  Plain
// arithmetic usable on the host, so a g++ harness checks the properties the
// kernel relies on (every slot filled exactly once, each lane's source inside
// the 1 KiB piece it lands in).
//
// gfx950's LDS serves a 16-byte read in four passes and a 16-byte write in
// eight; the placements below keep the lanes of every pass on distinct bank
// groups for the kernel's access patterns (measured with the LDS
// bank-conflict counter: no conflict cycles).
#pragma once
#include "plan.h"   // SG_HD

namespace specgen {

// V^T slices: the 16-byte half h (8 tokens) of dim row d of the slice of tile
// block kb sits at byte 512 (d / 16) + 256 (d & 1) + 32 ((d & 15) / 2) +
// 16 (h ^ (d & 1)) of the slice, with bit 5 flipped in odd blocks.  An
// operand read (dims 16 dt + ln over 16 lanes, one half, one block) and the
// E4M3 decode's writes (consecutive dims, one half) then hit distinct banks;
// the plain placement 2d + (h ^ bit 3 of d) took two passes per read.
SG_HD int v_pos(int d, int h, int kb) {
  return (512 * (d >> 4) + 256 * (d & 1) + 32 * ((d & 15) >> 1) + 16 * (h ^ (d & 1))) ^ (32 * (kb & 1));
}

// The inverse for a DMA: the dim row and half that v_pos places at byte
// 1024 i + 16 lane of the slice of block kb (piece i holds rows 32 i .. 32 i +
// 31, so the gather stays inside the piece).
SG_HD void v_slot_source(int i, int lane, int kb, int* d, int* h) {
  const int o = (16 * lane) ^ (32 * (kb & 1));
  const int w = (o >> 8) & 1;
  *d = 32 * i + 16 * (o >> 9) + 2 * ((o >> 5) & 7) + w;
  *h = ((o >> 4) & 1) ^ w;
}

// E4M3 K decode at head_dim 128: lane L of a wave converts token row
// kdec_row(L) of its 8-row code piece, bf16 chunks c0 and c0 + 1 with c0 =
// kdec_c0(L).  Each 8 consecutive lanes (one pass of a 16-byte LDS write)
// take half of each of two adjacent rows, whose K swizzles differ in bit 0, so
// their writes fall on distinct bank groups (one row per 8 lanes took two
// passes per write).
SG_HD int kdec_row(int L) { return 2 * ((L >> 3) & 3) + ((L & 7) >> 2); }
SG_HD int kdec_c0(int L) { return 2 * (L & 3) + 8 * (((L & 7) >> 2) ^ (L >> 5)); }

}  // namespace specgen
