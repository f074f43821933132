// Host check of the matrix-core code layouts (kvq_layout.h), built by
// test_layout.py with the system C++ compiler.
//
// 1. For b = 1, 2, 4, 8 the key and value bit maps are bijections onto the
//    row / block bits, and the *_owner functions invert them.
// 2. Packing random codes with the inverse maps and unpacking one MFMA
//    operand the way the decode kernel does (shifts, ANDs, byte permutes,
//    byte tables) gives back each element's code times the operand's fixed
//    weight (per element pair at one bit).
// Prints "ok" and exits 0, or prints the first mismatch and exits 1.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <random>
#include <vector>

#include "kvq_layout.h"

using kvq::BitLoc;

static int fail(const char* what, int b, int a0, int a1, int a2) {
  std::printf("FAIL %s b=%d (%d, %d, %d)\n", what, b, a0, a1, a2);
  return 1;
}

static int check_bijections(int b) {
  // keys: one token row of 4*b dwords
  std::vector<int> seen(4 * b * 32, 0);
  for (int c = 0; c < 128; ++c)
    for (int p = 0; p < b; ++p) {
      const BitLoc l = kvq::key_bit(c, p, b);
      if (l.word < 0 || l.word >= 4 * b || l.bit < 0 || l.bit >= 32) return fail("key_bit range", b, c, p, 0);
      if (seen[l.word * 32 + l.bit]++) return fail("key_bit collision", b, c, p, 0);
      int c2, p2;
      kvq::key_bit_owner(l.word, l.bit, b, c2, p2);
      if (c2 != c || p2 != p) return fail("key_bit_owner", b, c, p, 0);
      // the lane group that reads row dwords [b*g, b*g + b) owns the channel
      if (l.word / b != ((c >> 3) & 3)) return fail("key lane group", b, c, p, 0);
    }
  // values: one 32-token block of 128*b dwords
  std::vector<int> vseen(128 * b * 32, 0);
  for (int r = 0; r < 32; ++r)
    for (int c = 0; c < 128; ++c)
      for (int p = 0; p < b; ++p) {
        const BitLoc l = kvq::value_bit(r, c, p, b);
        if (l.word < 0 || l.word >= 128 * b || l.bit < 0 || l.bit >= 32) return fail("value_bit range", b, r, c, p);
        if (vseen[l.word * 32 + l.bit]++) return fail("value_bit collision", b, r, c, p);
        int r2, c2, p2;
        kvq::value_bit_owner(l.word, l.bit, b, r2, c2, p2);
        if (r2 != r || c2 != c || p2 != p) return fail("value_bit_owner", b, r, c, p);
        // lane L = c%16 + 16*kg reads dwords [2b*L, 2b*L + 2b)
        const int kg = (r & 15) >> 2;
        if (l.word / (2 * b) != (c & 15) + 16 * kg) return fail("value lane", b, r, c, p);
      }
  return 0;
}

// value of an fp16 bit pattern (subnormals and normals, non-negative)
static double half_value(uint32_t h) {
  const int e = (h >> 10) & 31, m = h & 1023;
  if (e == 0) return std::ldexp((double)m, -24);
  return std::ldexp(1.0 + m / 1024.0, e - 15);
}

static uint32_t perm(uint32_t src0, uint32_t src1, uint32_t sel) {
  uint8_t bytes[8];
  std::memcpy(bytes, &src1, 4);
  std::memcpy(bytes + 4, &src0, 4);
  uint32_t out = 0;
  for (int k = 0; k < 4; ++k) {
    const int s = (sel >> (8 * k)) & 0xFF;
    const uint32_t v = s < 8 ? bytes[s] : s == 0x0C ? 0u : 0xFFu;
    out |= v << (8 * k);
  }
  return out;
}

// The 8 halves of key operand kb of lane group g, unpacked as the kernel does.
static void key_operand(const uint32_t* row, int b, int g, int kb, uint32_t w[4]) {
  const uint32_t* x = row + b * g;
  if (b == 1) {
    const int sh = 4 * kb - 6;
    const uint32_t src = sh > 0 ? x[0] >> sh : x[0] << -sh;
    for (int i = 0; i < 4; ++i) w[i] = src & (0x10001u << (6 + i));
  } else if (b == 2) {
    const uint32_t v = x[kb >> 1];
    const int k = kb & 1;
    const uint32_t y1 = k ? v >> 2 : v << 6, y2 = k ? v >> 6 : v << 2;
    w[0] = y1 & 0x00C000C0u;
    w[1] = y1 & 0x03000300u;
    w[2] = y2 & 0x00C000C0u;
    w[3] = y2 & 0x03000300u;
  } else if (b == 4) {
    const uint32_t v = x[kb];
    w[0] = (v << 4) & 0x00F000F0u;
    w[1] = v & 0x00F000F0u;
    w[2] = (v >> 4) & 0x00F000F0u;
    w[3] = (v >> 8) & 0x00F000F0u;
  } else {
    for (int h = 0; h < 2; ++h) {
      w[2 * h] = perm(0u, x[2 * kb + h], 0x0C010C00u);
      w[2 * h + 1] = perm(0u, x[2 * kb + h], 0x0C030C02u);
    }
  }
}

// The 8 halves of value operand mb of lane L, as the kernel builds them.
static void value_operand(const uint32_t* blk, int b, int L, int mb, uint32_t w[4]) {
  const uint32_t* x = blk + 2 * b * L;
  if (b == 1) {
    const int sh = 4 * (mb & 3) - 6;
    const uint32_t src = sh > 0 ? x[mb >> 2] >> sh : x[mb >> 2] << -sh;
    for (int i = 0; i < 4; ++i) w[i] = src & (0x10001u << (6 + i));
  } else if (b == 2) {
    const uint32_t half_of[4] = {0x0000u, 0x3C00u, 0x4000u, 0x4200u};
    const uint32_t v = x[mb >> 1] >> (16 * (mb & 1));
    for (int j = 0; j < 2; ++j) {
      const uint32_t byte = (v >> (8 * j)) & 0xFF;
      for (int k = 0; k < 2; ++k)
        w[2 * j + k] = half_of[(byte >> (4 * k)) & 3] | (half_of[(byte >> (4 * k + 2)) & 3] << 16);
    }
  } else if (b == 4) {
    const uint32_t v = x[mb];
    w[0] = (v << 4) & 0x00F000F0u;
    w[1] = v & 0x00F000F0u;
    w[2] = (v >> 4) & 0x00F000F0u;
    w[3] = (v >> 8) & 0x00F000F0u;
  } else {
    for (int h = 0; h < 2; ++h) {
      w[2 * h] = perm(0u, x[2 * mb + h], 0x0C010C00u);
      w[2 * h + 1] = perm(0u, x[2 * mb + h], 0x0C030C02u);
    }
  }
}

static int check_operands(int b, std::mt19937& rng) {
  const int maxc = (1 << b) - 1;
  // keys: one token row
  uint8_t kc[128];
  for (int c = 0; c < 128; ++c) kc[c] = rng() % (maxc + 1);
  std::vector<uint32_t> row(4 * b, 0);
  for (int w = 0; w < 4 * b; ++w)
    for (int q = 0; q < 32; ++q) {
      int c, p;
      kvq::key_bit_owner(w, q, b, c, p);
      row[w] |= (uint32_t)((kc[c] >> p) & 1) << q;
    }
  // unit and per-element weight of each width (the kernel folds the weight
  // into the query and the unit into the fp32 scale)
  const int unit = b <= 2 ? 6 - 24 : b == 4 ? 4 - 24 : -24;
  for (int g = 0; g < 4; ++g)
    for (int kb = 0; kb < 4; ++kb) {
      uint32_t w[4];
      key_operand(row.data(), b, g, kb, w);
      for (int e = 0; e < 8; ++e) {
        const uint32_t h = (w[e >> 1] >> (16 * (e & 1))) & 0xFFFF;
        const int pair = e >> 1;
        const double weight = b == 1 ? std::ldexp(1.0, pair) : b == 2 ? ((pair & 1) ? 4.0 : 1.0) : 1.0;
        const double want = kc[32 * kb + 8 * g + e] * weight * std::ldexp(1.0, unit);
        if (half_value(h) != want) return fail("key operand", b, g, kb, e);
        // the top code bit stays at mantissa position 9 or lower (a subnormal)
        if (h >> 10) return fail("key operand not subnormal", b, g, kb, e);
      }
    }
  // values: one 32-token block
  std::vector<uint8_t> vc(32 * 128);
  for (auto& v : vc) v = rng() % (maxc + 1);
  std::vector<uint32_t> blk(128 * b, 0);
  for (int w = 0; w < 128 * b; ++w)
    for (int q = 0; q < 32; ++q) {
      int r, c, p;
      kvq::value_bit_owner(w, q, b, r, c, p);
      blk[w] |= (uint32_t)((vc[r * 128 + c] >> p) & 1) << q;
    }
  // 1-bit operands carry the key-style pair weight 2^i and unit 2^-18 (the
  // kernel folds 2^-i into the weights p); 2-bit table halves are exact codes
  const double vunit = b == 2 ? 1.0 : std::ldexp(1.0, b == 1 ? -18 : b == 4 ? -20 : -24);
  for (int L = 0; L < 64; ++L)
    for (int mb = 0; mb < 8; ++mb) {
      uint32_t w[4];
      value_operand(blk.data(), b, L, mb, w);
      for (int e = 0; e < 8; ++e) {
        const uint32_t h = (w[e >> 1] >> (16 * (e & 1))) & 0xFFFF;
        const int r = kvq::value_token(L >> 4, e), c = 16 * mb + (L & 15);
        const double vweight = b == 1 ? std::ldexp(1.0, e >> 1) : 1.0;
        if (half_value(h) != vc[r * 128 + c] * vweight * vunit) return fail("value operand", b, L, mb, e);
        if (b == 1 && (h >> 10)) return fail("value operand not subnormal", b, L, mb, e);
      }
    }
  return 0;
}

int main() {
  std::mt19937 rng(12345);
  for (int b : {1, 2, 4, 8}) {
    if (check_bijections(b)) return 1;
    for (int rep = 0; rep < 20; ++rep)
      if (check_operands(b, rng)) return 1;
  }
  std::printf("ok\n");
  return 0;
}
