// Matrix-core decode attention for caches with 1- or 2-bit keys and values
// and four query heads per kv head (gfx950, v_mfma_f32_16x16x32_f16).
//
// Same result as the vector kernel: softmax(q K^T / sqrt(d)) V over the
// dequantized cache (Introduction: scaled dot-product attention), split-K
// over tokens with an online softmax in base 2.  At one or two bits a token
// of one kv head carries 64-96 bytes but 2 * 4 * 128 multiply-adds, more than
// the vector ALUs can retire at HBM speed, so both contractions go to the
// matrix cores with every product exact and fp32 accumulation:
//
//   scores:  S^T[t][col] = sum_c code[t][c] * Q'[c][col] + sum_c z[c] * q~[c]
//     A = key codes as exact fp16 0/1 (or 0/2 for the high bit plane),
//     B = Q' = q~ (.) s split into fp16 hi + lo parts (two product terms,
//         each exact: q~ and s are fp16, their product fits two halves),
//     column col = 4*head + x: x = 0, 2 carry hi, x = 1, 3 carry lo; adding
//     the neighbour column gives hi + lo in every lane of the head.
//     The zero-point term uses A = z broadcast over tokens and B = q~.
//     q~ = q * 2^-e with |q~| < 1 keeps every fp16 operand finite; the scale
//     2^e * log2(e) / sqrt(d) is applied to the fp32 result.
//   values:  O^T[c][col] = sum_t code[t][c] * P'[t][col] (+ z term on VALU)
//     A = value codes (exact fp16), B = P' = p * s_v split hi / lo,
//     column col = 4*head + value group: a lane of the score layout already
//     holds p for the 8 tokens its B fragment needs (no transpose); output
//     columns whose group differs from the channel's are discarded.
//
// Packed bits become operands with one AND per element pair: a set bit at
// mantissa position w of a half is the exact fp16 subnormal 2^(w - 24).
// The key-side weights 2^w depend only on the channel and are folded into
// q~ once per decode; the value-side weights are split into a per-token-pair
// part folded into the value scales and a per-channel-block part applied to
// the accumulators at the end; the common 2^-24 goes into the fp32 scales.
// The layouts that place the bits are in kvq_layout.h.
#include <hip/hip_runtime.h>

#include "decode_common.h"
#include "kvq_internal.h"
#include "kvq_layout.h"

namespace kvq {
namespace {

using namespace dec;

typedef _Float16 h2_t __attribute__((ext_vector_type(2)));
typedef _Float16 h8_t __attribute__((ext_vector_type(8)));
typedef float f4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u4_t __attribute__((ext_vector_type(4)));

constexpr int kGQ = 4;
constexpr int kQRow = 80;  // dwords per Q' row in LDS: 64 + 16 of padding against bank conflicts

__device__ __forceinline__ h2_t u2h(uint32_t v) { return __builtin_bit_cast(h2_t, v); }
__device__ __forceinline__ uint32_t h2u(h2_t v) { return __builtin_bit_cast(uint32_t, v); }

// One MFMA operand (8 halves) from the bits of 4-channel block blk4 in x
// (bit plane `plane`): element pair i sits at bits (s, s + 16) with
// s = pair_bit(blk4, 2i), and a single AND leaves each half equal to
// bit * 2^(w - 24), an exact fp16 subnormal, with weight
// w = 4*(blk4 & 1) + i + plane.  The other operand or the output carries
// the inverse weight, so no multiply per element is needed.
__device__ __forceinline__ h8_t unpack8(uint32_t x, int blk4, int plane) {
  const uint32_t src = blk4 < 2 ? (plane ? x << 1 : x) : (plane ? x >> 7 : x >> 8);
  const int base = 4 * (blk4 & 1) + plane;
  u4_t w;
#pragma unroll
  for (int i = 0; i < 4; ++i) w[i] = src & (0x10001u << (base + i));
  return __builtin_bit_cast(h8_t, w);
}

__device__ __forceinline__ f4_t mfma(h8_t a, h8_t b, f4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

// Maximum over the four lane rows (lanes l, l^16, l^32, l^48) with the
// gfx950 row-swap permutes.
__device__ __forceinline__ float max_across_rows(float v) {
  const uint32_t u = __builtin_bit_cast(uint32_t, v);
  const auto s32 = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  v = fmaxf(__builtin_bit_cast(float, (uint32_t)s32[0]), __builtin_bit_cast(float, (uint32_t)s32[1]));
  const uint32_t w = __builtin_bit_cast(uint32_t, v);
  const auto s16 = __builtin_amdgcn_permlane16_swap(w, w, false, false);
  return fmaxf(__builtin_bit_cast(float, (uint32_t)s16[0]), __builtin_bit_cast(float, (uint32_t)s16[1]));
}

__device__ __forceinline__ float pick4(const float (&v)[kGQ], int i) {
  return i == 0 ? v[0] : i == 1 ? v[1] : i == 2 ? v[2] : v[3];
}

// Everything one 32-token block reads from memory.
template <int BK, int BV>
struct BlockData {
  uint32_t s;          // key scales of channels 2*lane, 2*lane+1 (this block's key group)
  uint32_t z;          // key zero-points of the same channels
  uint32_t kx[2][BK];  // key codes of tokens 16*mb + (lane & 15)
  uint32_t vx[2 * BV]; // value codes of this lane
  uint2 s01, s23, z01, z23;  // value scales / zeros of this lane's tokens and group
};

template <int BK, int BV>
__device__ __forceinline__ void load_block(const DecodeArgs& a, const uint8_t* blk, int j, int sub, int lane,
                                           int gsel, int ng, BlockData<BK, BV>& o) {
  const int col = lane & 15, row = lane >> 4;
  const uint8_t* kmeta = blk + a.km + (size_t)j * 2 * kHeadDim * 2;
  o.s = reinterpret_cast<const uint32_t*>(kmeta)[lane];
  o.z = reinterpret_cast<const uint32_t*>(kmeta + kHeadDim * 2)[lane];
  const int tok = j * a.gk + sub * 32;
#pragma unroll
  for (int mb = 0; mb < 2; ++mb) {
    const uint32_t* kr =
        reinterpret_cast<const uint32_t*>(blk + a.kc + (size_t)(tok + 16 * mb + col) * 16 * BK) + BK * row;
    if constexpr (BK == 1) {
      o.kx[mb][0] = kr[0];
    } else {
      const uint2 v = *reinterpret_cast<const uint2*>(kr);
      o.kx[mb][0] = v.x;
      o.kx[mb][1] = v.y;
    }
  }
  const int vb = tok / 32;
  const uint32_t* vr = reinterpret_cast<const uint32_t*>(blk + a.vc + (size_t)vb * 512 * BV) + lane * 2 * BV;
  if constexpr (BV == 1) {
    const uint2 v = *reinterpret_cast<const uint2*>(vr);
    o.vx[0] = v.x;
    o.vx[1] = v.y;
  } else {
    const uint4 v = *reinterpret_cast<const uint4*>(vr);
    o.vx[0] = v.x; o.vx[1] = v.y; o.vx[2] = v.z; o.vx[3] = v.w;
  }
  const uint8_t* vmb = blk + a.vm + (size_t)vb * 128 * ng;
  o.s01 = *reinterpret_cast<const uint2*>(vmb + value_meta_s(gsel, 4 * row));
  o.s23 = *reinterpret_cast<const uint2*>(vmb + value_meta_s(gsel, 16 + 4 * row));
  o.z01 = *reinterpret_cast<const uint2*>(vmb + value_meta_z(gsel, 4 * row, ng));
  o.z23 = *reinterpret_cast<const uint2*>(vmb + value_meta_z(gsel, 16 + 4 * row, ng));
}

template <int BK, int BV>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void decode_mfma_kernel(DecodeArgs a) {
  __shared__ uint32_t q_lds[kWaves][(2 * kGQ + 1) * kQRow];  // Q' hi rows, lo rows, key zero-points
  __shared__ float qp_lds[kWaves][kHeadDim * kGQ];  // fp16 tail split only
  __shared__ float p_lds[kWaves][32 * kGQ];         // fp16 tail split only
  __shared__ Reduce<kGQ> red;

  const Work wk = find_work(a);
  const DecodeSeq& S = a.seq[wk.si];
  const uint8_t* blk = a.arena + S.head0 + (uint64_t)wk.h * a.head_stride;
  // wave index as a scalar so that per-wave loop bounds stay in SGPRs
  const int lane = threadIdx.x & 63, wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);

  if (wk.sp >= S.nq) {  // fp16 tail tokens: vector path
    float qs0[kGQ], qs1[kGQ];
    load_q_scaled<kGQ>(a, S, wk.h, lane, qs0, qs1);
    State<kGQ> st;
    init_state<kGQ>(st);
    tail_split<kGQ>(a, S, blk, qs0, qs1, qp_lds[wv], p_lds[wv], st, lane, wv);
    stage_state<kGQ>(st, red, lane, wv);
    __syncthreads();
    write_record<kGQ>(a, S, wk.h, wk.sp, red);
    return;
  }

  const int col = lane & 15, row = lane >> 4;     // MFMA column, lane row
  const int hc = col >> 2, xc = col & 3, part = col & 1;
  const int ng = kHeadDim / a.gv, gsel = xc & (ng - 1);
  const uint16_t* qrow = a.q + ((size_t)S.seq * a.hq + (size_t)wk.h * kGQ) * kHeadDim;

  // q~ = q * 2^-e per head with max |q~| < 1.  For the code MFMA each lane's
  // channel pair (2*lane, 2*lane+1) also carries 2^-w, w = the bit weight of
  // those channels in the unpacked key operand.
  const float wq = ldexpf(1.f, -(4 * ((lane >> 4) & 1) + (lane & 3)));
  uint32_t qt[kGQ];
  float inv[kGQ], csc[kGQ];
#pragma unroll
  for (int g = 0; g < kGQ; ++g) {
    const uint32_t w = reinterpret_cast<const uint32_t*>(qrow + g * kHeadDim)[lane];
    const float q0 = h2f(w & 0xFFFF), q1 = h2f(w >> 16);
    const float mx = wave_max(fmaxf(fabsf(q0), fabsf(q1)));
    int e = 0;
    frexpf(mx, &e);
    inv[g] = ldexpf(1.f, -e);
    csc[g] = ldexpf(a.qscale, e + 24);  // undoes 2^-e and the 2^-24 of the code operand
    h2_t t;
    t.x = (_Float16)(q0 * inv[g] * wq);
    t.y = (_Float16)(q1 * inv[g] * wq);
    qt[g] = h2u(t);
  }
  const float cs = pick4(csc, hc);

  // B operand of the zero-point term: column (hc, hi) holds q~ of head hc
  h8_t bq[4];
  {
    const float iv = pick4(inv, hc);
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      const h8_t raw = *reinterpret_cast<const h8_t*>(qrow + hc * kHeadDim + 32 * kb + 8 * row);
#pragma unroll
      for (int e = 0; e < 8; ++e) bq[kb][e] = part ? (_Float16)0.f : (_Float16)((float)raw[e] * iv);
    }
  }

  float m = -__builtin_inff(), l = 0.f, zacc = 0.f;
  f4_t acc[8];
#pragma unroll
  for (int mb = 0; mb < 8; ++mb) acc[mb] = (f4_t){0.f, 0.f, 0.f, 0.f};

  const int t0 = wk.sp * a.split_tokens;
  const int t1 = min(S.Lq, t0 + a.split_tokens);
  uint32_t* ql = q_lds[wv];

  // This wave's 32-token blocks: key groups j0 + wv + kWaves*n, each of
  // gk/32 blocks.  Loads run one block ahead of the arithmetic.
  const int bpg = a.gk / 32;
  const int j0 = t0 / a.gk + wv, jend = t1 / a.gk;
  const int ngroups = j0 < jend ? (jend - j0 + kWaves - 1) / kWaves : 0;
  const int nblocks = ngroups * bpg;

  f4_t dz = {0.f, 0.f, 0.f, 0.f};
  h8_t bp[4];
  auto process = [&](const BlockData<BK, BV>& cur, int i) {
    if (i % bpg == 0) {
      // Q' = q~ (.) s of the block's key group, hi and lo halves, and the
      // group's zero-points, re-laid out through LDS
      wave_lds_sync();
#pragma unroll
      for (int g = 0; g < kGQ; ++g) {
        const h2_t q2 = u2h(qt[g]), s2 = u2h(cur.s);
        const h2_t hi = q2 * s2;
        const h2_t lo = __builtin_elementwise_fma(q2, s2, -hi);
        ql[g * kQRow + lane] = h2u(hi);
        ql[(kGQ + g) * kQRow + lane] = h2u(lo);
      }
      ql[2 * kGQ * kQRow + lane] = cur.z;
      wave_lds_sync();
      h8_t az[4];
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        bp[kb] = *reinterpret_cast<const h8_t*>(&ql[(part * kGQ + hc) * kQRow + 16 * kb + 4 * row]);
        az[kb] = *reinterpret_cast<const h8_t*>(&ql[2 * kGQ * kQRow + 16 * kb + 4 * row]);
      }
      dz = (f4_t){0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) dz = mfma(az[kb], bq[kb], dz);
      dz *= 0x1p-24f;  // to the scale of the code products
    }

    // scores of tokens 16*mb + 4*row + e of the block, e < 4
    f4_t d[2];
#pragma unroll
    for (int mb = 0; mb < 2; ++mb) {
      d[mb] = dz;
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int p = 0; p < BK; ++p) d[mb] = mfma(unpack8(cur.kx[mb][p], kb, p), bp[kb], d[mb]);
    }
    float sc[8];
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float v = d[mb][e];
        sc[4 * mb + e] = (v + dpp_mov<kQuadXor1>(0.f, v)) * cs;
      }

    // online softmax (base 2) for head hc over these 32 tokens
    float bm = sc[0];
#pragma unroll
    for (int t = 1; t < 8; ++t) bm = fmaxf(bm, sc[t]);
    bm = max_across_rows(bm);
    const float mnew = fmaxf(m, bm);
    const float alpha = __builtin_amdgcn_exp2f(m - mnew);
    m = mnew;
    float p[8], ps = 0.f;
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      p[t] = __builtin_amdgcn_exp2f(sc[t] - mnew);
      ps += p[t];
    }
    l = fmaf(l, alpha, ps);
    if (__builtin_amdgcn_ballot_w64(alpha != 1.f)) {
#pragma unroll
      for (int mb = 0; mb < 8; ++mb) acc[mb] *= alpha;
      zacc *= alpha;
    }

    // P' = p * s_v in hi / lo halves; element pair t = tokens of p[2t], p[2t+1]
    const uint32_t sv[4] = {cur.s01.x, cur.s01.y, cur.s23.x, cur.s23.y};
    const uint32_t zv[4] = {cur.z01.x, cur.z01.y, cur.z23.x, cur.z23.y};
    u4_t bhi, blo;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const h2_t ph = __builtin_bit_cast(h2_t, __builtin_amdgcn_cvt_pkrtz(p[2 * t], p[2 * t + 1]));
      const h2_t pl = __builtin_bit_cast(
          h2_t, __builtin_amdgcn_cvt_pkrtz(p[2 * t] - (float)ph.x, p[2 * t + 1] - (float)ph.y));
      // value scale times 2^-t, the inverse of the pair's bit weight
      const h2_t s2 = t == 0 ? u2h(sv[t]) : u2h(sv[t]) * (h2_t){(_Float16)(1.f / (1 << t)), (_Float16)(1.f / (1 << t))};
      const h2_t hi = ph * s2;
      const h2_t lo = __builtin_elementwise_fma(pl, s2, __builtin_elementwise_fma(ph, s2, -hi));
      bhi[t] = h2u(hi);
      blo[t] = h2u(lo);
      const h2_t z2 = u2h(zv[t]);
      zacc = fmaf(p[2 * t], (float)z2.x, fmaf(p[2 * t + 1], (float)z2.y, zacc));
    }
    const h8_t BH = __builtin_bit_cast(h8_t, bhi), BL = __builtin_bit_cast(h8_t, blo);
#pragma unroll
    for (int mb = 0; mb < 8; ++mb) {
#pragma unroll
      for (int p2 = 0; p2 < BV; ++p2) {
        const h8_t av = unpack8(cur.vx[(mb >> 2) * BV + p2], mb & 3, p2);
        acc[mb] = mfma(av, BH, acc[mb]);
        acc[mb] = mfma(av, BL, acc[mb]);
      }
    }
  };
  // block i of this wave: key group j0 + kWaves*(i / bpg), 32-token part i % bpg
  auto load = [&](int i, BlockData<BK, BV>& o) {
    load_block<BK, BV>(a, blk, j0 + kWaves * (i / bpg), i % bpg, lane, gsel, ng, o);
  };

  // Three buffers, loads two blocks ahead of the arithmetic.  The loads are
  // unconditional (past the end they re-read the last block) so every path
  // through the loop has the same loads in flight and the memory waits stay
  // exact.
  if (nblocks > 0) {
    const int last = nblocks - 1;
    BlockData<BK, BV> b0, b1, b2;
    load(0, b0);
    load(min(1, last), b1);
    for (int i = 0; i < nblocks; i += 3) {
      load(min(i + 2, last), b2);
      process(b0, i);
      if (i + 1 >= nblocks) break;
      load(min(i + 3, last), b0);
      process(b1, i + 1);
      if (i + 2 >= nblocks) break;
      load(min(i + 4, last), b1);
      process(b2, i + 2);
    }
  }

  // sums over the lane rows; the lanes of one head agree on m and l
  l += __shfl_xor(l, 16);
  l += __shfl_xor(l, 32);
  zacc += __shfl_xor(zacc, 16);
  zacc += __shfl_xor(zacc, 32);
#pragma unroll
  for (int mb = 0; mb < 8; ++mb) {
    if (xc == (16 * mb) / a.gv) {
#pragma unroll
      for (int e = 0; e < 4; ++e)  // undo the channel block's bit weight 2^(4*(mb & 1)) and the 2^-24
        red.acc[wv][hc * kHeadDim + 16 * mb + 4 * row + e] = fmaf(acc[mb][e], (mb & 1) ? 0x1p20f : 0x1p24f, zacc);
    }
  }
  if (row == 0 && xc == 0) {
    red.m[wv][hc] = m;
    red.l[wv][hc] = l;
  }
  __syncthreads();
  write_record<kGQ>(a, S, wk.h, wk.sp, red);
}

template <int BK, int BV>
int launch_t(const DecodeArgs& a, void* stream) {
  hipLaunchKernelGGL((decode_mfma_kernel<BK, BV>), dim3(a.total_wg), dim3(64 * kWaves), 0, (hipStream_t)stream, a);
  return (int)hipGetLastError();
}

}  // namespace

bool matrix_decode_supported(int bk, int bv, int gq, int gv) {
  return gq == kGQ && (bk == 1 || bk == 2) && (bv == 1 || bv == 2) && gv >= 32;
}

int launch_decode_matrix(const DecodeArgs& a, int bk, int bv, void* stream) {
  if (a.total_wg <= 0) return 0;
  if (bk == 1 && bv == 1) return launch_t<1, 1>(a, stream);
  if (bk == 1 && bv == 2) return launch_t<1, 2>(a, stream);
  if (bk == 2 && bv == 1) return launch_t<2, 1>(a, stream);
  if (bk == 2 && bv == 2) return launch_t<2, 2>(a, stream);
  return (int)hipErrorInvalidValue;
}

}  // namespace kvq
