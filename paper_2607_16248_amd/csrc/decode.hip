// Single-token decode attention over the packed low-bit KV cache (gfx950).
//
// out = softmax(q K^T / sqrt(d)) V for every query head (Introduction: the
// scaled dot-product attention the decoder runs at each step), with K and V
// dequantized in registers straight from the packed codes.
//
// Split-K over tokens (flash-decoding): each workgroup owns one
// (sequence, kv head, token range) and keeps an online softmax in base 2 for
// the Hq/Hkv query heads that read that kv head; a merge pass combines the
// per-split (max, sum, accumulator) records.  The packed codes carry no
// matrix-core-sized work (each token is a rank-GQ matrix-vector product), so
// everything runs on the vector ALUs:
//   - key scales are folded into the query once per key group,
//       q'_c = q_c * s_c * log2(e)/sqrt(d),   bias = sum_c q_c * z_c * log2(e)/sqrt(d),
//     so a score is bias + sum_c q'_c * code_c;
//   - values are dequantized per element as fma(code, s, z) and accumulated;
//   - wave-wide max and sum use DPP row operations and the row broadcasts.
#include <hip/hip_runtime.h>

#include "decode_common.h"
#include "kvq_internal.h"

namespace kvq {
namespace {

using namespace dec;

// Key row half (64 channels): 8*B bytes = 2*B dwords.
template <int B>
__device__ __forceinline__ void load_key_half(const uint8_t* row, uint32_t (&w)[2 * B]) {
  if constexpr (B == 1) {
    const uint2 v = *reinterpret_cast<const uint2*>(row);
    w[0] = v.x; w[1] = v.y;
  } else {
#pragma unroll
    for (int i = 0; i < B / 2; ++i) {
      const uint4 v = reinterpret_cast<const uint4*>(row)[i];
      w[4 * i] = v.x; w[4 * i + 1] = v.y; w[4 * i + 2] = v.z; w[4 * i + 3] = v.w;
    }
  }
}

// Value bits of 8 consecutive channels (8*B bits) of one token row.
template <int B>
__device__ __forceinline__ uint64_t load_value8(const uint8_t* row, int cc) {
  if constexpr (B == 1) return row[cc];
  else if constexpr (B == 2) return reinterpret_cast<const uint16_t*>(row)[cc];
  else if constexpr (B == 4) return reinterpret_cast<const uint32_t*>(row)[cc];
  else return reinterpret_cast<const uint64_t*>(row)[cc];
}

template <int BK, int BV, int GQ>
__device__ __forceinline__ void packed_group(const DecodeArgs& a, const DecodeSeq& S, int h, int j,
                                             const float (&qs0)[GQ], const float (&qs1)[GQ],
                                             float* qp, float* p_lds, State<GQ>& st, const int (&lim)[GQ],
                                             int glim, int lane) {
  constexpr int QS = QStride<GQ>::value;
  // the packed segment (head region or page) holding key group j, and the
  // group's first token in it
  int tj;
  const uint8_t* blk = a.arena + packed_seg(a.pm, S.head0, a.head_stride, S.seq, h, j * a.gk, tj);
  // scales and zeros of the key group: this lane's channels 2*lane, 2*lane+1
  const uint32_t* km = reinterpret_cast<const uint32_t*>(blk + a.km + (size_t)(tj / a.gk) * 2 * kHeadDim * 2);
  const uint32_t sw = km[lane], zw = km[kHeadDim / 2 + lane];
  const float s0 = h2f(sw & 0xFFFF), s1 = h2f(sw >> 16), z0 = h2f(zw & 0xFFFF), z1 = h2f(zw >> 16);
  float bias[GQ];
#pragma unroll
  for (int g = 0; g < GQ; ++g) {
    qp[(2 * lane) * QS + g] = qs0[g] * s0;
    qp[(2 * lane + 1) * QS + g] = qs1[g] * s1;
    bias[g] = fmaf(qs0[g], z0, qs1[g] * z1);
  }
#pragma unroll
  for (int g = 0; g < GQ; ++g) bias[g] = wave_sum(bias[g]);
  wave_lds_sync();

  const int tl = lane >> 1, half = lane & 1;
  const int tq = lane >> 4, cc = lane & 15;
  const int ng = kHeadDim / a.gv, vg = (cc * 8) / a.gv;
  for (int pass = 0; pass < a.gk / 32; ++pass) {
    const int tbase = j * a.gk + pass * 32;  // position in the sequence
    const int tseg = tj + pass * 32;         // position in the packed segment
    // scores: lane pair (2t, 2t+1) splits token t's 128 channels in halves
    uint32_t kw[2 * BK];
    load_key_half<BK>(blk + a.kc + (size_t)(tseg + tl) * 16 * BK + half * 8 * BK, kw);
    float sig[GQ];
#pragma unroll
    for (int g = 0; g < GQ; ++g) sig[g] = 0.f;
    constexpr int PER = 32 / BK;
    constexpr uint32_t MASK = (1u << BK) - 1u;
#pragma unroll
    for (int w = 0; w < 2 * BK; ++w) {
#pragma unroll
      for (int e = 0; e < PER; ++e) {
        const float code = (float)((kw[w] >> (e * BK)) & MASK);
        const float* qv = qp + (half * 64 + w * PER + e) * QS;
#pragma unroll
        for (int g = 0; g < GQ; ++g) sig[g] = fmaf(qv[g], code, sig[g]);
      }
    }
#pragma unroll
    for (int g = 0; g < GQ; ++g) sig[g] += dpp_mov<kQuadXor1>(0.f, sig[g]) + bias[g];
    if (tbase + 32 > glim) {  // tokens past a chunk query's position
#pragma unroll
      for (int g = 0; g < GQ; ++g)
        if (tbase + tl >= lim[g]) sig[g] = -__builtin_inff();
    }
    softmax_pass<GQ, true>(st, sig, half, tl, p_lds);
    wave_lds_sync();

    // values: lane (tq, cc) owns channels 8cc..8cc+7 for tokens tq, tq+4, ...
#pragma unroll 2
    for (int tt = tq; tt < 32; tt += 4) {
      const int t = tseg + tt;
      const uint32_t meta = reinterpret_cast<const uint32_t*>(blk + a.vm)[(size_t)t * ng + vg];
      const float sv = h2f(meta & 0xFFFF), zv = h2f(meta >> 16);
      const uint64_t vb = load_value8<BV>(blk + a.vc + (size_t)t * 16 * BV, cc);
      const float* pp = p_lds + tt * GQ;
      float pg[GQ];
#pragma unroll
      for (int g = 0; g < GQ; ++g) pg[g] = pp[g];
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const float v = fmaf((float)((uint32_t)(vb >> (k * BV)) & ((1u << BV) - 1u)), sv, zv);
#pragma unroll
        for (int g = 0; g < GQ; ++g) st.acc[g][k] = fmaf(pg[g], v, st.acc[g][k]);
      }
    }
    wave_lds_sync();
  }
}

template <int BK, int BV, int GQ>
__global__ __launch_bounds__(256) void decode_split_kernel(DecodeArgs a) {
  constexpr int QS = QStride<GQ>::value;
  __shared__ float qp_lds[kWaves][kHeadDim * QS];
  __shared__ float p_lds[kWaves][32 * GQ];
  __shared__ Reduce<GQ> red;

  const Work wk = find_work<true>(a);
  const DecodeSeq& S = a.seq[wk.si];
  const uint8_t* blk = a.arena + S.head0 + (uint64_t)wk.h * a.head_stride;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;

  float qs0[GQ], qs1[GQ];
  load_q_scaled<GQ, true>(a, S, wk.h, wk.rg, lane, qs0, qs1);
  State<GQ> st;
  init_state<GQ>(st);

  float* qp = qp_lds[wv];
  float* pl = p_lds[wv];
  if (wk.sp < S.nq) {
    const int t0 = wk.sp * a.split_tokens;
    const int t1 = min(S.Lq, t0 + a.split_tokens);
    int lim[GQ];
    row_limits<GQ>(a, S, wk.h, wk.rg, lim);
    const int glim = group_limit(a, S, wk.rg);
    for (int j = t0 / a.gk + wv; j < t1 / a.gk; j += kWaves)
      packed_group<BK, BV, GQ>(a, S, wk.h, j, qs0, qs1, qp, pl, st, lim, glim, lane);
  } else {
    tail_split<GQ, true>(a, S, wk.h, wk.rg, blk, qs0, qs1, qp, pl, st, lane, wv);
  }
  stage_state<GQ>(st, red, lane, wv);
  __syncthreads();
  write_record<GQ, true>(a, S, wk.h, wk.rg, wk.sp, red);
}

// One workgroup per (sequence, query head, 32-channel slice): thread
// (part, c) folds the records of splits part, part + 8, ... into a running
// (max, denominator, channel c numerator), loading U records at a time, U the
// smallest of 4, 5, 8, 9 and 17 for which one memory round trip covers all
// splits (up to 32, 40, 64, 72 or 136: a power of two of packed splits and
// the fp16-tail split fit; loads past the last split would re-read it); the
// eight parts then meet in LDS.  Four slices per head spread a head's records
// over four compute units.
constexpr int kMergeParts = 8;
constexpr int kMergeSlice = 32;
constexpr int kMergeSlices = kHeadDim / kMergeSlice;
constexpr int kMergeThreads = kMergeParts * kMergeSlice;

template <int U>
__device__ __forceinline__ void merge_fold(const float* base, size_t step, int n, int part, int c, float& M,
                                           float& D, float& A) {
  for (int i0 = part; i0 < n; i0 += kMergeParts * U) {
    float mv[U], lv[U], av[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = i0 + kMergeParts * u;
      const float* r = base + (size_t)min(i, n - 1) * step;
      mv[u] = r[0];
      lv[u] = r[1];
      av[u] = r[4 + c];
    }
    float mx = M;
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (i0 + kMergeParts * u < n) mx = fmaxf(mx, mv[u]);
    // M = -inf on the first batch: f = 0.  A split that saw no token of a
    // chunk query's row has m = -inf (l = 0, acc = 0); while every record so
    // far is such a split, mx = -inf and nothing is added.
    const bool none = mx == -__builtin_inff();
    const float f = none ? 1.f : __builtin_amdgcn_exp2f(M - mx);
    D *= f;
    A *= f;
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (i0 + kMergeParts * u < n) {
        const float w = none ? 0.f : __builtin_amdgcn_exp2f(mv[u] - mx);
        D = fmaf(w, lv[u], D);
        A = fmaf(w, av[u], A);
      }
    M = mx;
  }
}

__global__ __launch_bounds__(kMergeThreads) void merge_kernel(MergeArgs a) {
  __shared__ float sm[kMergeParts], sl[kMergeParts], sa[kMergeParts][kMergeSlice];
  const int head = blockIdx.x / kMergeSlices, slice = blockIdx.x % kMergeSlices;
  const int si = head / a.hq, hq = head % a.hq;
  const MergeSeq& S = a.seq[si];
  const int tid = threadIdx.x, cs = tid % kMergeSlice, part = tid / kMergeSlice;
  const int c = slice * kMergeSlice + cs;
  float* o = a.out + ((size_t)S.seq * a.hq + hq) * kHeadDim;
  const int n = S.nsplit;
  if (n == 0) {
    if (tid < kMergeSlice) o[c] = 0.f;
    return;
  }
  const float* base = a.ws + ((size_t)S.ws_base * a.hq + hq) * kRecFloats;
  const size_t step = (size_t)a.hq * kRecFloats;
  float M = -__builtin_inff(), D = 0.f, A = 0.f;
  if (n <= kMergeParts * 4) merge_fold<4>(base, step, n, part, c, M, D, A);
  else if (n <= kMergeParts * 5) merge_fold<5>(base, step, n, part, c, M, D, A);
  else if (n <= kMergeParts * 8) merge_fold<8>(base, step, n, part, c, M, D, A);
  else if (n <= kMergeParts * 9) merge_fold<9>(base, step, n, part, c, M, D, A);
  else merge_fold<17>(base, step, n, part, c, M, D, A);
  if (cs == 0) {
    sm[part] = M;
    sl[part] = D;
  }
  sa[part][cs] = A;
  __syncthreads();
  if (tid < kMergeSlice) {
    float mx = sm[0];
#pragma unroll
    for (int p = 1; p < kMergeParts; ++p) mx = fmaxf(mx, sm[p]);
    float den = 0.f, num = 0.f;
#pragma unroll
    for (int p = 0; p < kMergeParts; ++p) {
      // a part without splits, or without a visible token, has sm = -inf:
      // w = 0 (every row sees at least one token, so mx is finite)
      const float w = __builtin_amdgcn_exp2f(sm[p] - mx);
      den = fmaf(w, sl[p], den);
      num = fmaf(w, sa[p][cs], num);
    }
    o[c] = num / den;
  }
}

template <int BK, int BV, int GQ>
int launch_t(const DecodeArgs& a, void* stream) {
  hipLaunchKernelGGL((decode_split_kernel<BK, BV, GQ>), dim3(a.total_wg), dim3(64 * kWaves), 0,
                     (hipStream_t)stream, a);
  return (int)hipGetLastError();
}

template <int BK, int BV>
int launch_gq(const DecodeArgs& a, int gq, void* stream) {
  switch (gq) {
    case 1: return launch_t<BK, BV, 1>(a, stream);
    case 2: return launch_t<BK, BV, 2>(a, stream);
    case 4: return launch_t<BK, BV, 4>(a, stream);
    case 5: return launch_t<BK, BV, 5>(a, stream);
    case 8: return launch_t<BK, BV, 8>(a, stream);
    default: return (int)hipErrorInvalidValue;
  }
}

template <int BK>
int launch_bv(const DecodeArgs& a, int bv, int gq, void* stream) {
  switch (bv) {
    case 1: return launch_gq<BK, 1>(a, gq, stream);
    case 2: return launch_gq<BK, 2>(a, gq, stream);
    case 4: return launch_gq<BK, 4>(a, gq, stream);
    case 8: return launch_gq<BK, 8>(a, gq, stream);
    default: return (int)hipErrorInvalidValue;
  }
}

}  // namespace

int launch_decode(const DecodeArgs& a, int bk, int bv, int gq, void* stream) {
  if (a.total_wg <= 0) return 0;
  switch (bk) {
    case 1: return launch_bv<1>(a, bv, gq, stream);
    case 2: return launch_bv<2>(a, bv, gq, stream);
    case 4: return launch_bv<4>(a, bv, gq, stream);
    case 8: return launch_bv<8>(a, bv, gq, stream);
    default: return (int)hipErrorInvalidValue;
  }
}

int launch_merge(const MergeArgs& a, void* stream) {
  if (a.nseq <= 0) return 0;
  hipLaunchKernelGGL(merge_kernel, dim3(a.nseq * a.hq * kMergeSlices), dim3(kMergeThreads), 0, (hipStream_t)stream, a);
  return (int)hipGetLastError();
}

}  // namespace kvq
