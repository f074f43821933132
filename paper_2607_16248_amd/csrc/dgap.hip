// DGAP's logit-side runtime step (gfx950): features of the quantized
// logits, the risk detector, the top-K window and, on risky rows, the
// corrector and the sparse merge (Methodology: "DGAP Overview" online
// restoration framework, "Distribution-Risk Detector", "Selective Top-K
// Distribution Corrector"; the feature and MLP readings are stated in
// include/dgap.h).
//
// Two launches per call, both latency-bound at batch 1:
//   scan    one workgroup per (row, 2048-logit chunk): the chunk's max m and
//           its sums of e^(z-m), (m-z) e^(z-m) and e^(2(z-m)), and the chunk's
//           own top-K (a chunk's K largest contain every global winner that
//           falls in it) by radix selection over unique 64-bit keys;
//   finish  one workgroup per row: the log-sum-exp and entropy from the
//           chunk sums, the global top-K from the chunks' candidates (again
//           by radix selection), its order by rank counting, the 12
//           features, the detector and, when r > tau, the corrector over the
//           window and the in-place merge.
//
// Keys: the high 32 bits order the fp32 logits (sign-flipped bit patterns),
// the low 32 bits hold ~index, so that among equal logits the lower index
// is the larger key.  Keys are unique, so "the K largest keys" is exactly
// the window the paper selects with ties broken by index.
#include <hip/hip_runtime.h>

#include "decode_common.h"
#include "kvq_internal.h"

namespace kvq {
namespace {

using dec::dpp_mov;
using dec::kBcast15;
using dec::kBcast31;
using dec::kHalfMirror;
using dec::kMirror;
using dec::kQuadXor1;
using dec::kQuadXor2;
using dec::wave_max;
using dec::wave_sum;

constexpr int kScanThreads = 256;
constexpr int kScanItems = kDgapChunk / kScanThreads;  // logits per thread in a chunk
constexpr int kFinishThreads = 1024;
static_assert(32 * kFinishThreads == kDgapMaxCandidates, "the largest finish kernel holds every candidate");

__device__ __forceinline__ uint32_t order_bits(float f) {
  const uint32_t u = __builtin_bit_cast(uint32_t, f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float from_order_bits(uint32_t o) {
  return __builtin_bit_cast(float, (o & 0x80000000u) ? (o & 0x7FFFFFFFu) : ~o);
}
__device__ __forceinline__ uint64_t make_key(float v, uint32_t idx) {
  return ((uint64_t)order_bits(v) << 32) | (uint64_t)(~idx);
}
__device__ __forceinline__ float key_value(uint64_t k) { return from_order_bits((uint32_t)(k >> 32)); }
__device__ __forceinline__ uint32_t key_index(uint64_t k) { return ~(uint32_t)k; }

// Inclusive prefix sum over the 64 lanes of a wave: shifts by 1, 2, 4, 8
// within each 16-lane row (lanes without a source add 0), then the row
// totals through row broadcasts 15 and 31.  No LDS round trips.
__device__ __forceinline__ uint32_t wave_prefix_sum(uint32_t v) {
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xF, 0xF, false);  // row_shr:1
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xF, 0xF, false);  // row_shr:2
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xF, 0xF, false);  // row_shr:4
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xF, 0xF, false);  // row_shr:8
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xA, 0xF, false);  // row_bcast:15
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xC, 0xF, false);  // row_bcast:31
  return v;
}

template <int CTRL, int ROW_MASK = 0xF>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t old, uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)old, (int)v, CTRL, ROW_MASK, 0xF, false);
}

// Wave-wide maximum / minimum of unsigned 32-bit values (DPP, then lane 63).
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
  v = max(v, dpp_u32<kQuadXor1>(0u, v));
  v = max(v, dpp_u32<kQuadXor2>(0u, v));
  v = max(v, dpp_u32<kHalfMirror>(0u, v));
  v = max(v, dpp_u32<kMirror>(0u, v));
  v = max(v, dpp_u32<kBcast15, 0xA>(0u, v));
  v = max(v, dpp_u32<kBcast31, 0xC>(0u, v));
  return (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
}
__device__ __forceinline__ uint32_t wave_min_u32(uint32_t v) {
  v = min(v, dpp_u32<kQuadXor1>(~0u, v));
  v = min(v, dpp_u32<kQuadXor2>(~0u, v));
  v = min(v, dpp_u32<kHalfMirror>(~0u, v));
  v = min(v, dpp_u32<kMirror>(~0u, v));
  v = min(v, dpp_u32<kBcast15, 0xA>(~0u, v));
  v = min(v, dpp_u32<kBcast31, 0xC>(~0u, v));
  return (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
}

// Radix selection: the smallest key T with #{valid keys >= T} == want
// (keys unique and nonzero, at least `want` valid; 0 marks an empty slot).
// The search starts below the bits that the largest and the smallest valid
// key share (a window's candidates agree on their leading bits, which would
// otherwise pile into one histogram bucket), then takes digits of up to 8
// bits; a pass ends the search once the bucket holding the want-th key is
// needed whole.  LDS: hist[256], sel[3], ext[2 * 2 * NT / 64]; every thread
// of the block calls it.
template <int NT, int IPT>
__device__ uint64_t select_threshold(const uint64_t (&key)[IPT], int want, uint32_t* hist, uint32_t* sel,
                                     uint32_t* ext) {
  constexpr int kWavesPerBlock = NT / 64;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  // block-wide largest and smallest valid key
  uint64_t kmax = 0, kmin = ~0ull;
#pragma unroll
  for (int j = 0; j < IPT; ++j)
    if (key[j] != 0) {
      kmax = key[j] > kmax ? key[j] : kmax;
      kmin = key[j] < kmin ? key[j] : kmin;
    }
  {
    const uint32_t hmax = wave_max_u32((uint32_t)(kmax >> 32));
    const uint32_t lmax = wave_max_u32((uint32_t)(kmax >> 32) == hmax ? (uint32_t)kmax : 0u);
    const uint32_t hmin = wave_min_u32((uint32_t)(kmin >> 32));
    const uint32_t lmin = wave_min_u32((uint32_t)(kmin >> 32) == hmin ? (uint32_t)kmin : ~0u);
    if (lane == 0) {
      ext[4 * wv] = hmax;
      ext[4 * wv + 1] = lmax;
      ext[4 * wv + 2] = hmin;
      ext[4 * wv + 3] = lmin;
    }
  }
  __syncthreads();
  kmax = 0;
  kmin = ~0ull;
#pragma unroll
  for (int w = 0; w < kWavesPerBlock; ++w) {
    const uint64_t a = ((uint64_t)ext[4 * w] << 32) | ext[4 * w + 1];
    const uint64_t b = ((uint64_t)ext[4 * w + 2] << 32) | ext[4 * w + 3];
    kmax = a > kmax ? a : kmax;
    kmin = b < kmin ? b : kmin;
  }
  if (kmax == kmin) return kmax;  // a single valid key
  const int top = 63 - __builtin_clzll(kmax ^ kmin);  // highest bit that differs
  int width = min(8, top + 1), shift = top + 1 - width;
  uint64_t prefix = top == 63 ? 0 : kmax >> (top + 1);
  int rem = want;
  for (;;) {
    for (int i = tid; i < 256; i += NT) hist[i] = 0;
    __syncthreads();
    const uint32_t mask = (1u << width) - 1u;
#pragma unroll
    for (int j = 0; j < IPT; ++j) {
      const uint64_t k = key[j];
      if (k != 0 && (shift + width == 64 || (k >> (shift + width)) == prefix))
        atomicAdd(&hist[(uint32_t)(k >> shift) & mask], 1u);
    }
    __syncthreads();
    if (tid < 64) {
      // lane l holds buckets 255 - 4l .. 252 - 4l (descending)
      uint32_t c[4], own = 0;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        c[i] = hist[255 - 4 * tid - i];
        own += c[i];
      }
      uint32_t before = wave_prefix_sum(own) - own;  // keys in the buckets above this lane's
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if (before < (uint32_t)rem && before + c[i] >= (uint32_t)rem) {
          sel[0] = 255 - 4 * tid - i;
          sel[1] = before;
          sel[2] = c[i];
        }
        before += c[i];
      }
    }
    __syncthreads();
    const uint32_t digit = sel[0], above = sel[1], inbucket = sel[2];
    prefix = (prefix << width) | digit;
    rem -= (int)above;
    __syncthreads();  // sel and hist are rewritten by the next pass
    if ((int)inbucket == rem || shift == 0) return prefix << shift;
    width = min(8, shift);
    shift -= width;
  }
}

// Block sums of three values over kScanThreads threads (four waves).
__device__ __forceinline__ void block_sum4x3(float& a, float& b, float& c, float* red) {
  a = wave_sum(a);
  b = wave_sum(b);
  c = wave_sum(c);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    red[w] = a;
    red[4 + w] = b;
    red[8 + w] = c;
  }
  __syncthreads();
  a = (red[0] + red[1]) + (red[2] + red[3]);
  b = (red[4] + red[5]) + (red[6] + red[7]);
  c = (red[8] + red[9]) + (red[10] + red[11]);
  __syncthreads();
}
__device__ __forceinline__ float block_max4(float v, float* red) {
  v = wave_max(v);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  const float m = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  __syncthreads();
  return m;
}

__global__ __launch_bounds__(kScanThreads) void dgap_scan_kernel(DgapArgs a) {
  __shared__ uint32_t hist[256], sel[4], ext[4 * kScanThreads / 64];
  __shared__ float red[12];
  const int row = blockIdx.x / a.nchunk, chunk = blockIdx.x % a.nchunk;
  const float* z = a.logits + (size_t)row * a.vocab;
  const int base = chunk * kDgapChunk;
  float v[kScanItems];
  uint64_t key[kScanItems];
  float m = -__builtin_inff();
#pragma unroll
  for (int j = 0; j < kScanItems; ++j) {
    const int i = base + j * kScanThreads + threadIdx.x;
    const bool in = i < a.vocab;
    v[j] = in ? z[i] : -__builtin_inff();
    key[j] = in ? make_key(v[j], (uint32_t)i) : 0;
    m = fmaxf(m, v[j]);
  }
  m = block_max4(m, red);
  float s = 0.f, t = 0.f, u = 0.f;
#pragma unroll
  for (int j = 0; j < kScanItems; ++j) {
    if (key[j] != 0) {
      const float e = expf(v[j] - m);
      s += e;
      t = fmaf(e, m - v[j], t);  // >= 0 term by term: the entropy needs no cancellation
      u = fmaf(e, e, u);
    }
  }
  block_sum4x3(s, t, u, red);
  float* st = a.ws_stats + ((size_t)row * a.nchunk + chunk) * 4;
  if (threadIdx.x == 0) {
    st[0] = m;
    st[1] = s;
    st[2] = t;
    st[3] = u;
  }
  // the chunk's top-K (all of it when the chunk is shorter)
  const int n = min(kDgapChunk, a.vocab - base);
  const int want = min(a.k, n);
  uint64_t* out = a.ws_cand + ((size_t)row * a.nchunk + chunk) * a.k;
  const uint64_t T = want < n ? select_threshold<kScanThreads, kScanItems>(key, want, hist, sel, ext) : 1;
  if (threadIdx.x == 0) sel[3] = 0;
  __syncthreads();
#pragma unroll
  for (int j = 0; j < kScanItems; ++j)
    if (key[j] != 0 && key[j] >= T) {
      const uint32_t slot = atomicAdd(&sel[3], 1u);
      if (slot < (uint32_t)want) out[slot] = key[j];  // exactly `want` keys pass
    }
  for (int i = want + threadIdx.x; i < a.k; i += kScanThreads) out[i] = 0;  // empty slots
}

// IPT: candidate keys per thread (the launch picks the smallest of 8, 16, 32
// that holds chunks * K).
template <int IPT>
__global__ __launch_bounds__(kFinishThreads) void dgap_finish_kernel(DgapArgs a) {
  constexpr int kW1 = kDgapFeatures * kDgapMaxHidden, kC1 = (kDgapCandInputs + kDgapFeatures) * kDgapMaxHidden;
  __shared__ float wdet[kW1 + 2 * kDgapMaxHidden], wcor[kC1 + 2 * kDgapMaxHidden];
  __shared__ uint32_t hist[256], sel[4], ext[4 * kFinishThreads / 64];
  __shared__ uint64_t win[kDgapMaxK], skey[kDgapMaxK];
  __shared__ float stat[8];      // lse, H, sum p^2, r
  __shared__ float phi[kDgapFeatures];
  __shared__ float vsorted[kDgapMaxK];
  __shared__ float uphi[kDgapMaxHidden];
  const int row = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int K = a.k, ncand = a.nchunk * K;
  float* z = a.logits + (size_t)row * a.vocab;
  const int hd = a.hidden_det, hc = a.hidden_corr;

  // Every global load is issued first so that their latencies overlap: the
  // candidate keys, the MLP weights (three elements per thread of the
  // concatenation det_w1, det_b1, det_w2, corr_w1, corr_b1, corr_w2) and,
  // in wave 0, the statistics of the first 64 chunks.
  uint64_t key[IPT];
  const uint64_t* cand = a.ws_cand + (size_t)row * ncand;
#pragma unroll
  for (int j = 0; j < IPT; ++j) {
    const int i = j * kFinishThreads + tid;
    key[j] = i < ncand ? cand[i] : 0;
  }
  const int seg[6] = {kDgapFeatures * hd, hd, hd, (kDgapCandInputs + kDgapFeatures) * hc, hc, hc};
  const float* src[6] = {a.det_w1, a.det_b1, a.det_w2, a.corr_w1, a.corr_b1, a.corr_w2};
  float* dst[6] = {wdet, wdet + kW1, wdet + kW1 + kDgapMaxHidden, wcor, wcor + kC1, wcor + kC1 + kDgapMaxHidden};
  float wv3[3];
  int ws3[3], wo3[3];
#pragma unroll
  for (int r3 = 0; r3 < 3; ++r3) {
    int i = tid + r3 * kFinishThreads, sgi = 0;
    while (sgi < 6 && i >= seg[sgi]) i -= seg[sgi++];
    ws3[r3] = sgi;
    wo3[r3] = i;
    wv3[r3] = sgi < 6 ? src[sgi][i] : 0.f;
  }
  const float* st = a.ws_stats + (size_t)row * a.nchunk * 4;
  float4 st0 = make_float4(-__builtin_inff(), 0.f, 0.f, 0.f);
  if (wv == 0 && lane < a.nchunk) st0 = *reinterpret_cast<const float4*>(st + 4 * lane);
#pragma unroll
  for (int r3 = 0; r3 < 3; ++r3)
    if (ws3[r3] < 6) dst[ws3[r3]][wo3[r3]] = wv3[r3];

  // log-sum-exp, entropy and concentration from the chunk sums (wave 0)
  if (wv == 0) {
    float M = st0.x;
    for (int c = lane + 64; c < a.nchunk; c += 64) M = fmaxf(M, st[4 * c]);
    M = wave_max(M);
    const bool has0 = lane < a.nchunk;  // (lanes past the last chunk add nothing)
    float S = has0 ? expf(st0.x - M) * st0.y : 0.f;
    for (int c = lane + 64; c < a.nchunk; c += 64) S += expf(st[4 * c] - M) * st[4 * c + 1];
    S = wave_sum(S);
    const float lse = M + logf(S);
    // H = sum_i p_i (lse - z_i) = sum_chunks e^(m-lse) ((lse - m) s + sum_i e_i (m - z_i)),
    // every term non-negative
    const float f0 = has0 ? expf(st0.x - lse) : 0.f;
    float h = has0 ? f0 * fmaf(lse - st0.x, st0.y, st0.z) : 0.f, p2 = f0 * f0 * st0.w;
    for (int c = lane + 64; c < a.nchunk; c += 64) {
      const float f = expf(st[4 * c] - lse);
      h = fmaf(f, fmaf(lse - st[4 * c], st[4 * c + 1], st[4 * c + 2]), h);
      p2 = fmaf(f * f, st[4 * c + 3], p2);
    }
    h = wave_sum(h);
    p2 = wave_sum(p2);
    if (lane == 0) {
      stat[0] = lse;
      stat[1] = h;
      stat[2] = p2;
    }
  }

  // the global window: the K largest candidate keys, then their order
  const uint64_t T = select_threshold<kFinishThreads, IPT>(key, K, hist, sel, ext);
  if (tid == 0) sel[3] = 0;
  __syncthreads();
#pragma unroll
  for (int j = 0; j < IPT; ++j)
    if (key[j] != 0 && key[j] >= T) {
      const uint32_t slot = atomicAdd(&sel[3], 1u);
      if (slot < (uint32_t)K) win[slot] = key[j];  // exactly K keys pass
    }
  __syncthreads();
  {
    // rank of window entry c = #{larger entries}: four threads per entry
    const int c = tid >> 2, part = tid & 3;
    const uint64_t mine = c < K ? win[c] : 0;
    int rank = 0;
    if (c < K) {
      for (int j0 = part; j0 < K; j0 += 4 * 16) {  // 16 reads in flight
        uint64_t o[16];
#pragma unroll
        for (int u = 0; u < 16; ++u) o[u] = j0 + 4 * u < K ? win[j0 + 4 * u] : 0;
#pragma unroll
        for (int u = 0; u < 16; ++u) rank += o[u] > mine;
      }
    }
    // the four threads of an entry are one lane quad
    rank += (int)dpp_u32<kQuadXor1>(0u, (uint32_t)rank);
    rank += (int)dpp_u32<kQuadXor2>(0u, (uint32_t)rank);
    if (c < K && part == 0) {
      skey[rank] = mine;
      vsorted[rank] = key_value(mine);
    }
  }
  __syncthreads();

  // features (wave 0; four window entries per lane)
  const float lse = stat[0];
  if (wv == 0) {
    float P[4], vv[4];
    float mass = 0.f, top8 = 0.f, vsum = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int k = lane + 64 * i;
      vv[i] = k < K ? vsorted[k] : 0.f;
      P[i] = k < K ? expf(vv[i] - lse) : 0.f;
      mass += P[i];
      vsum += vv[i];
      if (k < 8) top8 += P[i];
    }
    mass = wave_sum(mass);
    top8 = wave_sum(top8);
    const float mean = wave_sum(vsum) / K;
    float var = 0.f, hk = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int k = lane + 64 * i;
      if (k < K) {
        var = fmaf(vv[i] - mean, vv[i] - mean, var);
        const float q = P[i] / mass;
        if (q > 0.f) hk -= q * logf(q);
      }
    }
    var = wave_sum(var) / K;
    hk = wave_sum(hk);
    if (lane == 0) {
      const float H = stat[1];
      float mg = vsorted[0] - vsorted[1];
      for (int k = 1; k < 7; ++k) mg = fminf(mg, vsorted[k] - vsorted[k + 1]);
      phi[0] = H;
      phi[1] = H / logf((float)a.vocab);
      phi[2] = vsorted[0] - lse;
      phi[3] = mass;
      phi[4] = top8;
      phi[5] = stat[2];
      phi[6] = vsorted[0] - vsorted[1];
      phi[7] = vsorted[1] - vsorted[2];
      phi[8] = (vsorted[0] - vsorted[K - 1]) / (float)(K - 1);
      phi[9] = mg;
      phi[10] = sqrtf(var);
      phi[11] = hk;
    }
  }
  __syncthreads();

  // detector: lane h is hidden unit h (wave 0)
  if (wv == 0) {
    float y = 0.f;
    if (lane < hd) {
      float acc = wdet[kW1 + lane];
#pragma unroll
      for (int i = 0; i < kDgapFeatures; ++i) acc = fmaf(phi[i], wdet[i * hd + lane], acc);
      y = fmaxf(acc, 0.f) * wdet[kW1 + kDgapMaxHidden + lane];
    }
    const float s = wave_sum(y) + a.det_b2;
    if (lane == 0) stat[3] = 1.f / (1.f + expf(-s));
  }
  __syncthreads();
  const float r = stat[3];
  const bool correct = r > a.tau;
  float* info = a.info ? a.info + (size_t)row * (kDgapInfoHead + 2 * K) : nullptr;

  if (correct) {
    // corrector: the phi part of hidden unit h's input is the same for every
    // candidate (wave 0 computes it); then four threads (a lane quad) per
    // candidate, 16 hidden units each
    if (wv == 0 && lane < hc) {
      float uh = wcor[kC1 + lane];
#pragma unroll
      for (int i = 0; i < kDgapFeatures; ++i) uh = fmaf(phi[i], wcor[(kDgapCandInputs + i) * hc + lane], uh);
      uphi[lane] = uh;
    }
    __syncthreads();
    const int k = tid >> 2, g = tid & 3;
    float part = 0.f, vk = 0.f;
    if (k < K) {
      vk = vsorted[k];
      const float xi[kDgapCandInputs] = {vk - vsorted[0], vk - lse, (float)k / (float)(K - 1),
                                         k > 0 ? vsorted[k - 1] - vk : 0.f, k + 1 < K ? vk - vsorted[k + 1] : 0.f};
      for (int h = 16 * g; h < min(hc, 16 * g + 16); ++h) {
        float acc = uphi[h];
#pragma unroll
        for (int i = 0; i < kDgapCandInputs; ++i) acc = fmaf(xi[i], wcor[i * hc + h], acc);
        part = fmaf(fmaxf(acc, 0.f), wcor[kC1 + kDgapMaxHidden + h], part);
      }
    }
    part += __builtin_bit_cast(float, dpp_u32<kQuadXor1>(0u, __builtin_bit_cast(uint32_t, part)));
    part += __builtin_bit_cast(float, dpp_u32<kQuadXor2>(0u, __builtin_bit_cast(uint32_t, part)));
    if (k < K && g == 0) {
      const float d = part + a.corr_b2;
      const uint32_t idx = key_index(skey[k]);
      if (idx < (uint32_t)a.vocab) z[idx] = vk + d;
      if (info) info[kDgapInfoHead + K + k] = d;
    }
  } else if (info) {
    for (int k = tid; k < K; k += kFinishThreads) info[kDgapInfoHead + K + k] = 0.f;
  }
  if (info) {
    for (int k = tid; k < K; k += kFinishThreads)
      info[kDgapInfoHead + k] = __builtin_bit_cast(float, key_index(skey[k]));
    if (tid < kDgapFeatures) info[4 + tid] = phi[tid];
    if (tid == 0) {
      info[0] = r;
      info[1] = correct ? 1.f : 0.f;
      info[2] = lse;
      info[3] = 0.f;
    }
  }
}

}  // namespace

int launch_dgap(const DgapArgs& a, int batch, void* stream) {
  hipLaunchKernelGGL(dgap_scan_kernel, dim3(batch * a.nchunk), dim3(kScanThreads), 0, (hipStream_t)stream, a);
  int e = (int)hipGetLastError();
  if (e) return e;
  const int ncand = a.nchunk * a.k;
  if (ncand <= 8 * kFinishThreads)
    hipLaunchKernelGGL(dgap_finish_kernel<8>, dim3(batch), dim3(kFinishThreads), 0, (hipStream_t)stream, a);
  else if (ncand <= 16 * kFinishThreads)
    hipLaunchKernelGGL(dgap_finish_kernel<16>, dim3(batch), dim3(kFinishThreads), 0, (hipStream_t)stream, a);
  else
    hipLaunchKernelGGL(dgap_finish_kernel<32>, dim3(batch), dim3(kFinishThreads), 0, (hipStream_t)stream, a);
  return (int)hipGetLastError();
}

}  // namespace kvq
