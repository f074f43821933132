// Device bit layouts of the packed codes.
//
// Two layouts exist per sequence, chosen when the cache is created:
//
//  canonical  key and value code rows of 16*b bytes per token, channel c at
//             row bits [c*b, c*b + b); value meta [t][128/Gv][(s, z)].
//             This is also the export image's order.
//
//  matrix     (caches read by the matrix-core decode kernel)
//    The codes one lane of a 16x16x32 MFMA operand needs (8 elements) sit
//    together in the lane's dwords, placed so that a few shifts and ANDs, a
//    byte permute or a table lookup turn them into the operand's halves.
//    key rows: 16*b bytes per token; lane group g (0..3) of the operand owns
//      row dwords [b*g, b*g + b) and channels c = 32*kb + 8*g + e (kb: the
//      operand's 32-channel block, e: its element 0..7).  Per width:
//      b = 1: dword g, bit pair_bit(kb, e) = 16*(e&1) + 8*(kb>>1) + 4*(kb&1)
//             + (e>>1): bits (s, s + 16) hold a consecutive element pair, one
//             AND after a shift per block makes two fp16 values;
//      b = 2: dword 2*g + (kb>>1), code bits at 8*(kb&1) + 2*(e>>1) + 16*(e&1):
//             two shifts and four ANDs place element pairs 0, 2 at mantissa
//             bits 6-7 and pairs 1, 3 at bits 8-9;
//      b = 4: dword 4*g + kb, nibble (e>>1) + 4*(e&1) (element pair i at
//             nibbles i, i + 4);
//      b = 8: dword 8*g + 2*kb + (e>>2), byte e&3.
//    value codes: blocks of 32 tokens, 512*b bytes each, in the lane order of
//      the MFMA A-operand of O^T = V^T P: lane L = c%16 + 16*kg holds 2*b
//      dwords; operand mb (channels 16*mb .. 16*mb + 15, channel c =
//      16*mb + c%16) has elements e' (0..7) for block tokens r = tau(8*kg + e'),
//      tau(8*kg + e') = 4*kg + e' for e' < 4 and 16 + 4*kg + (e' - 4) otherwise.
//      b = 1: dword mb >> 2, bit pair_bit(mb&3, e'): like 1-bit keys, element
//             pair i at bits (s, s + 16), s = 4*(mb&3) + i, so one shift and
//             four ANDs per operand make its halves;
//      b = 2: dword mb >> 1, bits 16*(mb&1) + 2*e': two bytes per operand,
//             each looked up in a 256-entry table of 4 halves;
//      b = 4: dword mb, nibble (e'>>1) + 4*(e'&1);
//      b = 8: dword 2*mb + (e'>>2), byte e'&3.
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

// Which caches the matrix-core decode kernel serves: 1- or 2-bit keys and
// values in any combination, or 4- or 8-bit keys and values in any
// combination; 1, 2, 4, 5 or 8 query heads per kv head (1 and 2 in the
// four-head layout with empty heads); value groups of at least 32 channels.
KVQ_HD constexpr bool matrix_bits(int bk, int bv) {
  return ((bk == 1 || bk == 2) && (bv == 1 || bv == 2)) || ((bk == 4 || bk == 8) && (bv == 4 || bv == 8));
}
KVQ_HD constexpr bool matrix_heads(int gq, int gk) {
  return (gq == 1 || gq == 2 || gq == 4 || gq == 5 || gq == 8) && gk % 32 == 0;
}
// Waves per SIMD its instantiations are compiled for: four for 1-bit keys
// and values with one 32-token block per key group, three for the other 1-
// and 2-bit four-head cases with one block per group, else two (registers).
// bpg = key_group / 32.
// gq = 16 or 32 names the chunk kernel with that many rows: three waves per
// SIMD for 16 rows of 1-bit values with 1- or 2-bit keys, else two.
KVQ_HD constexpr int chunk_waves(int bk, int bv, int rows) { return (rows == 16 && bv == 1 && bk <= 2) ? 3 : 2; }
// Row groups of 32 (two row halves sharing the unpacked operands) for 1- and
// 2-bit keys and values.
KVQ_HD constexpr bool chunk_rows32(int bk, int bv) { return bk <= 2 && bv <= 2; }
KVQ_HD constexpr int matrix_waves(int bk, int bv, int bpg, int gq) {
  return gq >= 16 ? chunk_waves(bk, bv, gq) : (gq > 4 || bk > 2 || bv > 2) ? 2 : bpg == 1 ? (bk + bv == 2 ? 4 : 3) : 2;
}

KVQ_HD inline int pair_bit(int blk4, int e) {
  return 16 * (e & 1) + 8 * (blk4 >> 1) + 4 * (blk4 & 1) + (e >> 1);
}

struct BitLoc {
  int word;  // dword index (within the key row, or within the value block)
  int bit;
};

// Dword (within the operand's dwords) and bit offset of element e (0..7)
// of a whole-code operand at 4 or 8 bits; field_elem inverts it.
KVQ_HD inline int elem_word(int e, int b) { return b == 8 ? e >> 2 : 0; }
KVQ_HD inline int elem_field(int e, int b) { return b == 8 ? e & 3 : (e >> 1) + 4 * (e & 1); }
KVQ_HD inline int field_elem(int w, int f, int b) { return b == 8 ? 4 * w + f : 2 * (f & 3) + (f >> 2); }

// Key code bit p of channel c (matrix layout): dword within the row, bit.
KVQ_HD inline BitLoc key_bit(int c, int p, int b) {
  const int kb = c >> 5, g = (c >> 3) & 3, e = c & 7;
  if (b == 1) return {g, pair_bit(kb, e)};
  if (b == 2) return {2 * g + (kb >> 1), 8 * (kb & 1) + 2 * (e >> 1) + 16 * (e & 1) + p};
  return {(b / 4) * (4 * g + kb) + elem_word(e, b), b * elem_field(e, b) + p};
}

// The channel and code bit that key row dword w, bit q holds.
KVQ_HD inline void key_bit_owner(int w, int q, int b, int& c, int& p) {
  int g, kb, e;
  if (b == 1) {
    g = w;
    kb = 2 * ((q >> 3) & 1) + ((q >> 2) & 1);
    e = 2 * (q & 3) + (q >> 4);
    p = 0;
  } else if (b == 2) {
    g = w >> 1;
    kb = 2 * (w & 1) + ((q >> 3) & 1);
    e = 2 * ((q >> 1) & 3) + (q >> 4);
    p = q & 1;
  } else {
    const int o = w / (b / 4);  // = 4*g + kb
    g = o >> 2;
    kb = o & 3;
    e = field_elem(w % (b / 4), q / b, b);
    p = q % b;
  }
  c = 32 * kb + 8 * g + e;
}

// Block token of value-operand element e' of K-group kg.
KVQ_HD inline int value_token(int kg, int e) { return e < 4 ? 4 * kg + e : 16 + 4 * kg + (e - 4); }

// Value code bit p of block token r (0..31), channel c (matrix layout):
// dword within the 32-token block, bit.
KVQ_HD inline BitLoc value_bit(int r, int c, int p, int b) {
  const int hi = r >> 4, r16 = r & 15;
  const int kg = r16 >> 2, e = (r16 & 3) + 4 * hi;
  const int mb = c >> 4;
  const int lane = (c & 15) + 16 * kg;
  if (b == 1) return {lane * 2 + (mb >> 2), pair_bit(mb & 3, e)};
  if (b == 2) return {lane * 4 + (mb >> 1), 16 * (mb & 1) + 2 * e + p};
  return {lane * 2 * b + (b / 4) * mb + elem_word(e, b), b * elem_field(e, b) + p};
}

// The block token, channel and code bit that value block dword w, bit q holds.
KVQ_HD inline void value_bit_owner(int w, int q, int b, int& r, int& c, int& p) {
  const int lane = w / (2 * b), o = w % (2 * b);
  int mb, e;
  if (b == 1) {
    mb = 4 * o + 2 * ((q >> 3) & 1) + ((q >> 2) & 1);
    e = 2 * (q & 3) + (q >> 4);
    p = 0;
  } else if (b == 2) {
    mb = 2 * o + (q >> 4);
    e = (q >> 1) & 7;
    p = q & 1;
  } else {
    mb = o / (b / 4);
    e = field_elem(o % (b / 4), q / b, b);
    p = q % b;
  }
  r = value_token(lane >> 4, e);
  c = 16 * mb + (lane & 15);
}

// Position of block token r in a value meta row: tau^-1, so that
// r = tau(pos) with tau(8*kg + e') = 4*kg + e' (e' < 4), 16 + 4*kg + e' - 4.
KVQ_HD inline int value_meta_pos(int r) { return 8 * ((r & 15) >> 2) + 4 * (r >> 4) + (r & 3); }

// Byte offsets of a value block's scale and zero of (group g, token r).
KVQ_HD inline int value_meta_s(int g, int r) { return (g * 32 + value_meta_pos(r)) * 2; }
KVQ_HD inline int value_meta_z(int g, int r, int ng) { return (ng * 32 + g * 32 + value_meta_pos(r)) * 2; }

}  // namespace kvq
