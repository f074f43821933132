// Device bit layouts of the packed codes.
//
// Two layouts exist per sequence, chosen when the cache is created:
//
//  canonical  key and value code rows of 16*b bytes per token, channel c at
//             row bits [c*b, c*b + b); value meta [t][128/Gv][(s, z)].
//             This is also the export image's order.
//
//  matrix     (caches read by the matrix-core decode kernel)
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
//    4- and 8-bit codes (the b = 4 and 8 variants of the above) are not split
//      into bit planes: a dword holds whole codes, 32/b fields of b bits, so
//      that the codes of one MFMA operand become its halves with one
//      instruction per pair.  Field f of a dword holds operand element
//      e = field_elem(f, b): b = 8, dword h of an 8-element operand holds
//      elements 4h + f at byte f; b = 4, the operand's single dword holds
//      element pair i at nibbles (i, i + 4).
//      keys: channel c = 32*kb + 8*g + e sits in row dword (b/4)*(4*g + kb)
//        + (b == 8 ? e >> 2 : 0);
//      values: lane L holds 2*b dwords, channel block mb in dwords
//        (b/4)*mb + (b == 8 ? e' >> 2 : 0) of the lane, e' as above.
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

// Whole-code (4- and 8-bit) operand layout: the dword (within the operand's
// b/4 dwords) and field of operand element e (0..7), and its inverse.
KVQ_HD inline int elem_word(int e, int b) { return b == 8 ? e >> 2 : 0; }
KVQ_HD inline int elem_field(int e, int b) { return b == 8 ? e & 3 : (e >> 1) + 4 * (e & 1); }
KVQ_HD inline int field_elem(int w, int f, int b) { return b == 8 ? 4 * w + f : 2 * (f & 3) + (f >> 2); }

// Key code bit of channel c, plane p (matrix layout).
KVQ_HD inline BitLoc key_bit(int c, int p, int b) {
  const int kb = c >> 5, g = (c >> 3) & 3, e = c & 7;
  if (b <= 2) return {g * b + p, pair_bit(kb, e)};
  return {(b / 4) * (4 * g + kb) + elem_word(e, b), b * elem_field(e, b) + p};
}

// Channel of field f of key row dword w (whole-code layouts).
KVQ_HD inline int key_field_channel(int w, int f, int b) {
  const int q = w / (b / 4), g = q >> 2, kb = q & 3;
  return 32 * kb + 8 * g + field_elem(w % (b / 4), f, b);
}

// Bit of value-operand element e' (0..7) of channel block m4 (0..3) in its dword.
KVQ_HD inline int value_elem_bit(int m4, int e) { return 8 * m4 + e; }

// Block token of value-operand element e' of K-group kg.
KVQ_HD inline int value_token(int kg, int e) { return e < 4 ? 4 * kg + e : 16 + 4 * kg + (e - 4); }

// Value code bit of block token r (0..31), channel c, plane p.
KVQ_HD inline BitLoc value_bit(int r, int c, int p, int b) {
  const int hi = r >> 4, r16 = r & 15;
  const int kg = r16 >> 2, e = (r16 & 3) + 4 * hi;
  const int mb = c >> 4, d = mb >> 2, m4 = mb & 3;
  const int lane = (c & 15) + 16 * kg;
  if (b <= 2) return {lane * 2 * b + d * b + p, value_elem_bit(m4, e)};
  return {lane * 2 * b + (b / 4) * mb + elem_word(e, b), b * elem_field(e, b) + p};
}

// Block token and channel of field f of value block dword w (whole-code layouts).
KVQ_HD inline void value_field_loc(int w, int f, int b, int& r, int& c) {
  const int lane = w / (2 * b), q = w % (2 * b), mb = q / (b / 4);
  r = value_token(lane >> 4, field_elem(q % (b / 4), f, b));
  c = 16 * mb + (lane & 15);
}

// Position of block token r in a value meta row: tau^-1, so that
// r = tau(pos) with tau(8*kg + e') = 4*kg + e' (e' < 4), 16 + 4*kg + e' - 4.
KVQ_HD inline int value_meta_pos(int r) { return 8 * ((r & 15) >> 2) + 4 * (r >> 4) + (r & 3); }

// Byte offsets of a value block's scale and zero of (group g, token r).
KVQ_HD inline int value_meta_s(int g, int r) { return (g * 32 + value_meta_pos(r)) * 2; }
KVQ_HD inline int value_meta_z(int g, int r, int ng) { return (ng * 32 + g * 32 + value_meta_pos(r)) * 2; }

}  // namespace kvq
