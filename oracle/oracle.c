/*
 * CPU oracle for the packed low-bit KV-cache decode path.
 *
 * TEST INFRASTRUCTURE ONLY (tests, smoke check, CPU baseline of the
 * benchmark).  Plain, slow, fp64; no blocking, no fusion, no online softmax.
 * Shares no code with the HIP library.  Build flags keep IEEE semantics:
 * -ffp-contract=off and no fast-math.
 *
 * The paper fixes the attention computation (Introduction: softmax of the
 * scaled query-key scores times V) and the notion of b-bit keys and b-bit
 * values (Motivation, "Accuracy Loss under Aggressive KV Quantization",
 * Methodology paragraph), and says the cache stays at that precision for the
 * whole decode (Methodology, "DGAP Overview", online restoration framework).
 * It does not define the quantizer.  The reading implemented here:
 *   - asymmetric min-max: zero-point z = group minimum (an fp16 value),
 *     scale s = the smallest fp16 >= (max - min) / (2^b - 1),
 *     code = round-half-even((x - z) / s), dequantized value z + code * s;
 *     a constant group has s = 0 and all codes 0;
 *   - keys are grouped per channel over key_group consecutive tokens,
 *     values per token over value_group consecutive channels;
 *   - tokens are quantized a whole key group at a time once they are more
 *     than `window` tokens from the end; the rest stay fp16.
 */
#include "oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

double orc_half_value(uint16_t h) {
  int sign = h >> 15;
  int e = (h >> 10) & 0x1f;
  int m = h & 0x3ff;
  double v;
  if (e == 0)
    v = ldexp((double)m, -24);                 /* subnormal: m * 2^-24 */
  else if (e == 31)
    v = m ? NAN : INFINITY;
  else
    v = ldexp((double)(m | 0x400), e - 25);    /* (1024 + m) * 2^(e-15-10) */
  return sign ? -v : v;
}

/* Positive finite fp16 patterns 0x0001..0x7BFF increase with their value, so
 * the smallest one >= s is found by bisection with exact fp64 comparisons. */
int orc_half_ceil(double s, uint16_t* out) {
  if (!(s >= 0.0) || isinf(s)) return ORC_ERR_RANGE;
  if (s == 0.0) { *out = 0; return ORC_OK; }
  if (s > 65504.0) return ORC_ERR_RANGE;
  unsigned lo = 1, hi = 0x7BFF;                /* value(hi) = 65504 >= s */
  while (lo < hi) {
    unsigned mid = (lo + hi) / 2;
    if (orc_half_value((uint16_t)mid) >= s)
      hi = mid;
    else
      lo = mid + 1;
  }
  *out = (uint16_t)lo;
  return ORC_OK;
}

/* x - z is exact in fp64 for fp16 inputs, the scale is the smallest fp16 at
 * or above the fp64 quotient (which equals the smallest at or above the exact
 * quotient, as a nonzero gap between the two exceeds fp64 rounding), and
 * rint() rounds half to even under the default rounding mode. */
int orc_quantize_group(const uint16_t* x, long n, long stride, int bits,
                       uint16_t* s, uint16_t* z, uint8_t* codes) {
  if (n <= 0 || !(bits == 1 || bits == 2 || bits == 4 || bits == 8)) return ORC_ERR_ARG;
  double mn = INFINITY, mx = -INFINITY;
  uint16_t zb = 0;
  for (long i = 0; i < n; ++i) {
    double v = orc_half_value(x[i * stride]);
    if (!isfinite(v)) return ORC_ERR_RANGE;
    if (v < mn) { mn = v; zb = x[i * stride]; }
    if (v > mx) mx = v;
  }
  if (mn == 0.0) zb = 0;                       /* zero-point +0, never -0 */
  double qmax = (double)((1 << bits) - 1);
  uint16_t sb;
  if (orc_half_ceil((mx - mn) / qmax, &sb) != ORC_OK) return ORC_ERR_RANGE;
  double sv = orc_half_value(sb);
  for (long i = 0; i < n; ++i) {
    double r = 0.0;
    if (sv != 0.0) r = rint((orc_half_value(x[i * stride]) - mn) / sv);
    if (!(r >= 0.0 && r <= qmax)) return ORC_ERR_ARG;  /* cannot happen: s >= (max-min)/qmax */
    codes[i] = (uint8_t)r;
  }
  *s = sb;
  *z = zb;
  return ORC_OK;
}

long orc_quantized_len(long L, int key_group, int window) {
  long past = L - window;
  if (past <= 0) return 0;
  return (past / key_group) * key_group;
}

static int valid_args(long L, int d, int bk, int bv, int gk, int gv, int window) {
  int okb = (bk == 1 || bk == 2 || bk == 4 || bk == 8) && (bv == 1 || bv == 2 || bv == 4 || bv == 8);
  return okb && L >= 0 && d > 0 && d % 8 == 0 && gk > 0 && gv > 0 && d % gv == 0 && window >= 0;
}

/* Canonical image of one (sequence, kv head), in this order, no padding:
 *   1. key codes   [Lq][d*bk/8]: token rows; the code of channel c occupies
 *      row bits [c*bk, c*bk + bk), least significant bit first, where row bit
 *      i is bit (i mod 8) of byte i/8;
 *   2. key meta    [Lq/gk][2][d] fp16: the group's d scales, then d zeros;
 *   3. value codes [Lq][d*bv/8], packed like the key codes;
 *   4. value meta  [Lq][d/gv][2] fp16: (scale, zero) per value group;
 *   5. key tail    [L-Lq][d] fp16, then 6. value tail [L-Lq][d] fp16.
 * fp16 values are stored little-endian. */
size_t orc_head_bytes(long L, int d, int bk, int bv, int gk, int gv, int window) {
  if (!valid_args(L, d, bk, bv, gk, gv, window)) return 0;
  long Lq = orc_quantized_len(L, gk, window);
  size_t n = 0;
  n += (size_t)Lq * d * bk / 8;
  n += (size_t)(Lq / gk) * 2 * d * 2;
  n += (size_t)Lq * d * bv / 8;
  n += (size_t)Lq * (d / gv) * 2 * 2;
  n += (size_t)(L - Lq) * d * 2 * 2;
  return n;
}

static void put_code(uint8_t* row, long c, int bits, unsigned code) {
  for (int k = 0; k < bits; ++k) {
    long bit = c * bits + k;
    if ((code >> k) & 1u) row[bit >> 3] |= (uint8_t)(1u << (bit & 7));
  }
}

static unsigned get_code(const uint8_t* row, long c, int bits) {
  unsigned code = 0;
  for (int k = 0; k < bits; ++k) {
    long bit = c * bits + k;
    code |= (unsigned)((row[bit >> 3] >> (bit & 7)) & 1u) << k;
  }
  return code;
}

static void put_half(uint8_t* p, uint16_t h) { p[0] = (uint8_t)(h & 0xff); p[1] = (uint8_t)(h >> 8); }
static uint16_t get_half(const uint8_t* p) { return (uint16_t)(p[0] | (p[1] << 8)); }

int orc_build_head(const uint16_t* K, const uint16_t* V, long L, long rs, int d,
                   int bk, int bv, int gk, int gv, int window, uint8_t* out) {
  if (!valid_args(L, d, bk, bv, gk, gv, window) || gk > 4096 || d > 4096) return ORC_ERR_ARG;
  long Lq = orc_quantized_len(L, gk, window);
  size_t rowk = (size_t)d * bk / 8, rowv = (size_t)d * bv / 8;
  uint8_t* kc = out;
  uint8_t* km = kc + (size_t)Lq * rowk;
  uint8_t* vc = km + (size_t)(Lq / gk) * 2 * d * 2;
  uint8_t* vm = vc + (size_t)Lq * rowv;
  uint8_t* kt = vm + (size_t)Lq * (d / gv) * 2 * 2;
  uint8_t* vt = kt + (size_t)(L - Lq) * d * 2;
  memset(out, 0, orc_head_bytes(L, d, bk, bv, gk, gv, window));

  uint8_t codes[4096];
  uint16_t s, z;
  for (long j = 0; j < Lq / gk; ++j) {
    for (int c = 0; c < d; ++c) {
      int st = orc_quantize_group(K + (j * gk) * rs + c, gk, rs, bk, &s, &z, codes);
      if (st != ORC_OK) return st;
      put_half(km + ((size_t)j * 2 * d + c) * 2, s);
      put_half(km + ((size_t)j * 2 * d + d + c) * 2, z);
      for (int i = 0; i < gk; ++i) put_code(kc + (size_t)(j * gk + i) * rowk, c, bk, codes[i]);
    }
  }
  for (long t = 0; t < Lq; ++t) {
    for (int g = 0; g < d / gv; ++g) {
      int st = orc_quantize_group(V + t * rs + (long)g * gv, gv, 1, bv, &s, &z, codes);
      if (st != ORC_OK) return st;
      put_half(vm + ((size_t)t * (d / gv) + g) * 4, s);
      put_half(vm + ((size_t)t * (d / gv) + g) * 4 + 2, z);
      for (int i = 0; i < gv; ++i) put_code(vc + (size_t)t * rowv, (long)g * gv + i, bv, codes[i]);
    }
  }
  for (long t = Lq; t < L; ++t) {
    for (int c = 0; c < d; ++c) {
      put_half(kt + ((size_t)(t - Lq) * d + c) * 2, K[t * rs + c]);
      put_half(vt + ((size_t)(t - Lq) * d + c) * 2, V[t * rs + c]);
    }
  }
  return ORC_OK;
}

/* z + code * s is exact in fp64: code < 2^8 and s has 11 significant bits,
 * and every fp16 value is a multiple of 2^-24 below 2^16 in magnitude. */
int orc_dequant_head(const uint8_t* img, long L, int d, int bk, int bv, int gk, int gv,
                     int window, double* Khat, double* Vhat) {
  if (!valid_args(L, d, bk, bv, gk, gv, window)) return ORC_ERR_ARG;
  long Lq = orc_quantized_len(L, gk, window);
  size_t rowk = (size_t)d * bk / 8, rowv = (size_t)d * bv / 8;
  const uint8_t* kc = img;
  const uint8_t* km = kc + (size_t)Lq * rowk;
  const uint8_t* vc = km + (size_t)(Lq / gk) * 2 * d * 2;
  const uint8_t* vm = vc + (size_t)Lq * rowv;
  const uint8_t* kt = vm + (size_t)Lq * (d / gv) * 2 * 2;
  const uint8_t* vt = kt + (size_t)(L - Lq) * d * 2;
  for (long t = 0; t < Lq; ++t) {
    long j = t / gk;
    for (int c = 0; c < d; ++c) {
      double s = orc_half_value(get_half(km + ((size_t)j * 2 * d + c) * 2));
      double z = orc_half_value(get_half(km + ((size_t)j * 2 * d + d + c) * 2));
      Khat[t * d + c] = z + (double)get_code(kc + (size_t)t * rowk, c, bk) * s;
      int g = c / gv;
      double sv = orc_half_value(get_half(vm + ((size_t)t * (d / gv) + g) * 4));
      double zv = orc_half_value(get_half(vm + ((size_t)t * (d / gv) + g) * 4 + 2));
      Vhat[t * d + c] = zv + (double)get_code(vc + (size_t)t * rowv, c, bv) * sv;
    }
  }
  for (long t = Lq; t < L; ++t) {
    for (int c = 0; c < d; ++c) {
      Khat[t * d + c] = orc_half_value(get_half(kt + ((size_t)(t - Lq) * d + c) * 2));
      Vhat[t * d + c] = orc_half_value(get_half(vt + ((size_t)(t - Lq) * d + c) * 2));
    }
  }
  return ORC_OK;
}

/* softmax(q K^T / sqrt(d)) V for each query head, directly from the
 * definition: all scores, their maximum, the exponentials, their sum. */
int orc_attention(const uint16_t* q, const double* Khat, const double* Vhat, long L,
                  int Hq, int Hkv, int d, double* out, double* weights) {
  if (Hq <= 0 || Hkv <= 0 || Hq % Hkv != 0 || d <= 0 || L < 0) return ORC_ERR_ARG;
  int gq = Hq / Hkv;
  double inv_sqrt_d = 1.0 / sqrt((double)d);
  int status = ORC_OK;
#pragma omp parallel for schedule(dynamic, 1)
  for (int h = 0; h < Hq; ++h) {
    const double* Kh = Khat + (size_t)(h / gq) * L * d;
    const double* Vh = Vhat + (size_t)(h / gq) * L * d;
    double* o = out + (size_t)h * d;
    for (int c = 0; c < d; ++c) o[c] = 0.0;
    if (L == 0) continue;
    double* w = (double*)malloc((size_t)L * sizeof(double));
    if (!w) { status = ORC_ERR_ARG; continue; }
    double m = -INFINITY;
    for (long t = 0; t < L; ++t) {
      double acc = 0.0;
      for (int c = 0; c < d; ++c) acc += orc_half_value(q[(size_t)h * d + c]) * Kh[t * d + c];
      w[t] = acc * inv_sqrt_d;
      if (w[t] > m) m = w[t];
    }
    double Z = 0.0;
    for (long t = 0; t < L; ++t) {
      w[t] = exp(w[t] - m);
      Z += w[t];
    }
    for (long t = 0; t < L; ++t) {
      for (int c = 0; c < d; ++c) o[c] += w[t] * Vh[t * d + c];
    }
    for (int c = 0; c < d; ++c) o[c] /= Z;
    if (weights)
      for (long t = 0; t < L; ++t) weights[(size_t)h * L + t] = w[t] / Z;
    free(w);
  }
  return status;
}

int orc_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}
