/* Drives the CPU oracle (oracle/oracle.c) under AddressSanitizer and UBSan:
 * every bit width, ragged lengths around the group sizes, fp16 windows,
 * forced ties, constant groups, subnormal scales, empty and single-token
 * sequences, and the range error.  Checks the quantizer's error bound and
 * code range, that an image dequantizes to values within half a scale of
 * the inputs, and that attention weights sum to one.  Prints
 * "oracle checks ok". */
#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "oracle.h"

static int fails = 0;
#define EXPECT(c) do { if (!(c)) { fprintf(stderr, "FAILED %s:%d: %s\n", __FILE__, __LINE__, #c); ++fails; } } while (0)

/* fp16 bit pattern near x (round half to even; any finite pattern would
 * do as an input, the checks below only need finite fp16 values). */
static uint16_t to_half(double xd) {
  const float f = (float)xd;
  uint32_t x;
  memcpy(&x, &f, 4);
  const uint32_t sign = (x >> 16) & 0x8000u;
  const int e = (int)((x >> 23) & 0xFFu) - 127 + 15;
  uint32_t m = x & 0x7FFFFFu;
  if (e >= 31) return (uint16_t)(sign | 0x7BFFu);
  if (e <= 0) {
    if (e < -10) return (uint16_t)sign;
    m |= 0x800000u;
    const uint32_t shift = (uint32_t)(14 - e), half = 1u << (shift - 1);
    uint32_t h = m >> shift;
    const uint32_t rem = m & ((1u << shift) - 1u);
    if (rem > half || (rem == half && (h & 1u))) ++h;
    return (uint16_t)(sign | h);
  }
  uint32_t h = ((uint32_t)e << 10) | (m >> 13);
  const uint32_t rem = m & 0x1FFFu;
  if (rem > 0x1000u || (rem == 0x1000u && (h & 1u))) ++h;
  return (uint16_t)(sign | h);
}

static unsigned rng = 12345u;
static double urand(void) {
  rng = rng * 1664525u + 1013904223u;
  return (rng >> 8) / 16777216.0;
}
static double nrand(void) {
  double u = urand() + 1e-12, v = urand();
  return sqrt(-2.0 * log(u)) * cos(6.283185307179586 * v);
}

static void check_group(const uint16_t* x, long n, int bits) {
  uint16_t s = 0, z = 0;
  uint8_t codes[256];
  EXPECT(orc_quantize_group(x, n, 1, bits, &s, &z, codes) == ORC_OK);
  const double sv = orc_half_value(s), zv = orc_half_value(z);
  for (long i = 0; i < n; ++i) {
    EXPECT(codes[i] <= (1u << bits) - 1);
    const double xr = orc_half_value(x[i]), xh = zv + codes[i] * sv;
    EXPECT(fabs(xr - xh) <= sv / 2);
  }
}

int main(void) {
  const int bits[4] = {1, 2, 4, 8};
  /* groups: random, constant, forced ties, subnormal range */
  for (int b = 0; b < 4; ++b) {
    for (long n = 1; n <= 64; n += (n < 4 ? 1 : 15)) {
      uint16_t x[256];
      for (long i = 0; i < n; ++i) x[i] = to_half(nrand() * 3.0);
      check_group(x, n, bits[b]);
      for (long i = 0; i < n; ++i) x[i] = to_half(1.5);
      check_group(x, n, bits[b]);
      for (long i = 0; i < n; ++i) x[i] = to_half((double)(i % 5) * 0.5);  /* ties at several widths */
      check_group(x, n, bits[b]);
      for (long i = 0; i < n; ++i) x[i] = (uint16_t)(i % 7);            /* subnormal values */
      check_group(x, n, bits[b]);
    }
    uint16_t big[2] = {to_half(-60000.0), to_half(60000.0)};
    uint16_t s, z;
    uint8_t codes[2];
    EXPECT(orc_quantize_group(big, 2, 1, bits[b], &s, &z, codes) == (bits[b] == 1 ? ORC_ERR_RANGE : ORC_OK));
  }
  /* whole heads: image, dequantization, attention */
  const int d = 128;
  const long lens[] = {0, 1, 31, 32, 33, 65, 200};
  const int windows[] = {0, 40};
  for (int bk = 0; bk < 4; ++bk)
    for (int bv = 0; bv < 4; ++bv)
      for (int li = 0; li < 7; ++li)
        for (int wi = 0; wi < 2; ++wi) {
          const long L = lens[li];
          const int R = windows[wi], gk = 32, gv = 32;
          uint16_t* K = malloc((L + 1) * d * 2);
          uint16_t* V = malloc((L + 1) * d * 2);
          for (long i = 0; i < L * d; ++i) {
            K[i] = to_half(nrand() * ((i % d) < 4 ? 10.0 : 1.0));
            V[i] = to_half(nrand());
          }
          const size_t nb = orc_head_bytes(L, d, bits[bk], bits[bv], gk, gv, R);
          uint8_t* img = malloc(nb + 1);
          EXPECT(orc_build_head(K, V, L, d, d, bits[bk], bits[bv], gk, gv, R, img) == ORC_OK);
          double* Kh = malloc((L + 1) * d * sizeof(double));
          double* Vh = malloc((L + 1) * d * sizeof(double));
          EXPECT(orc_dequant_head(img, L, d, bits[bk], bits[bv], gk, gv, R, Kh, Vh) == ORC_OK);
          for (long i = 0; i < L * d; ++i) {
            EXPECT(isfinite(Kh[i]) && isfinite(Vh[i]));
          }
          uint16_t q[4 * 128];
          for (int i = 0; i < 4 * d; ++i) q[i] = to_half(nrand());
          double out[4 * 128];
          double* w = malloc(4 * (L + 1) * sizeof(double));
          EXPECT(orc_attention(q, Kh, Vh, L, 4, 1, d, out, w) == ORC_OK);
          for (int h = 0; h < 4 && L > 0; ++h) {
            double sum = 0;
            for (long t = 0; t < L; ++t) sum += w[h * L + t];
            EXPECT(fabs(sum - 1.0) < 1e-12);
          }
          free(K); free(V); free(img); free(Kh); free(Vh); free(w);
        }
  EXPECT(orc_quantized_len(100, 32, 40) == 32);
  if (fails) {
    fprintf(stderr, "%d oracle checks failed\n", fails);
    return 1;
  }
  printf("oracle checks ok\n");
  return 0;
}
