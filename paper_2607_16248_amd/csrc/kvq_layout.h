// Device bit layouts of the packed codes.
//
// Two layouts exist per sequence, chosen when the cache is created:
//
//  canonical  key and value code rows of 16*b bytes per token, channel c at
//             row bits [c*b, c*b + b); value meta [t][128/Gv][(s, z)].
//             This is also the export image's order.
//
//  matrix     (1- and 2-bit caches read by the matrix-core decode kernel)
//    key rows: still 16*b bytes per token, but permuted so that the 32
//      channels one lane of a 16x16x32 MFMA A-operand needs sit in one dword
//      per bit plane: channel c = 32*kb + 8*g + e (kb, g in 0..3, e in 0..7)
//      lives in dword b*g + p (bit plane p of its code) at bit
//      pair_bit(kb, e) = 16*(e&1) + 8*(kb>>1) + 4*(kb&1) + (e>>1).
//      Bits (pair_bit, pair_bit + 16) then hold a consecutive element pair,
//      which one AND turns into two fp16 values (exact subnormal powers of 2).
//    value codes: blocks of 32 tokens, 512*b bytes each, in the lane order of
//      the MFMA A-operand of O^T = V^T P: lane L = c%16 + 16*kg holds 2*b
//      dwords; dword d*b + p covers channel blocks mb = 4d + m4 (m4 in 0..3),
//      channel c = 16*mb + c%16, byte m4 holding the K-index elements e'
//      (0..7, bit e' of the byte), for block token r = tau(8*kg + e') where
//      tau(8*kg + e') = 4*kg + e' for e' < 4 and 16 + 4*kg + (e' - 4) otherwise.
//      One byte is one A operand (8 halves), looked up in a 256-entry table.
//    value meta: per 32-token block, scales s[g][pos(r)] then zeros
//      z[g][pos(r)] (fp16, g < 128/Gv, r < 32): 128*(128/Gv) bytes, the same
//      total as the canonical [t][g][(s, z)] order.  pos = tau^-1 puts the 8
//      tokens of K-group kg (lanes 16*kg .. 16*kg + 15) in 16 contiguous bytes,
//      in B-fragment element order.
//    key meta is [group][s[128], z[128]] in both layouts.
#pragma once

#include <stdint.h>

#ifdef __HIPCC__
#define KVQ_HD __host__ __device__
#else
#define KVQ_HD
#endif

namespace kvq {

KVQ_HD inline int pair_bit(int blk4, int e) {
  return 16 * (e & 1) + 8 * (blk4 >> 1) + 4 * (blk4 & 1) + (e >> 1);
}

struct BitLoc {
  int word;  // dword index (within the key row, or within the value block)
  int bit;
};

// Key code bit of channel c, plane p (matrix layout, b in {1, 2}).
KVQ_HD inline BitLoc key_bit(int c, int p, int b) {
  const int kb = c >> 5, g = (c >> 3) & 3, e = c & 7;
  return {g * b + p, pair_bit(kb, e)};
}

// Bit of value-operand element e' (0..7) of channel block m4 (0..3) in its dword.
KVQ_HD inline int value_elem_bit(int m4, int e) { return 8 * m4 + e; }

// Value code bit of block token r (0..31), channel c, plane p.
KVQ_HD inline BitLoc value_bit(int r, int c, int p, int b) {
  const int hi = r >> 4, r16 = r & 15;
  const int kg = r16 >> 2, e = (r16 & 3) + 4 * hi;
  const int mb = c >> 4, d = mb >> 2, m4 = mb & 3;
  const int lane = (c & 15) + 16 * kg;
  return {lane * 2 * b + d * b + p, value_elem_bit(m4, e)};
}

// Position of block token r in a value meta row: tau^-1, so that
// r = tau(pos) with tau(8*kg + e') = 4*kg + e' (e' < 4), 16 + 4*kg + e' - 4.
KVQ_HD inline int value_meta_pos(int r) { return 8 * ((r & 15) >> 2) + 4 * (r >> 4) + (r & 3); }

// Byte offsets of a value block's scale and zero of (group g, token r).
KVQ_HD inline int value_meta_s(int g, int r) { return (g * 32 + value_meta_pos(r)) * 2; }
KVQ_HD inline int value_meta_z(int g, int r, int ng) { return (ng * 32 + g * 32 + value_meta_pos(r)) * 2; }

}  // namespace kvq
