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
constexpr int kFinishItems = kDgapMaxCandidates / kFinishThreads;

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

// Radix selection: the smallest key T with #{valid keys >= T} == want
// (keys unique, at least `want` valid).  Eight-bit digits from the top; a
// pass ends the search once the bucket holding the want-th key is needed
// whole.  LDS: hist[256], sel[3]; every thread of the block calls it.
template <int NT, int IPT>
__device__ uint64_t select_threshold(const uint64_t (&key)[IPT], int want, uint32_t* hist, uint32_t* sel) {
  const int tid = threadIdx.x;
  uint64_t prefix = 0;
  int rem = want;
  for (int shift = 56;; shift -= 8) {
    for (int i = tid; i < 256; i += NT) hist[i] = 0;
    __syncthreads();
#pragma unroll
    for (int j = 0; j < IPT; ++j) {
      const uint64_t k = key[j];
      if (k != 0 && (shift == 56 || (k >> (shift + 8)) == prefix))
        atomicAdd(&hist[(uint32_t)(k >> shift) & 0xFFu], 1u);
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
      uint32_t before = own;  // inclusive scan over lanes, then exclusive
#pragma unroll
      for (int d = 1; d < 64; d <<= 1) {
        const uint32_t o = __shfl_up(before, d);
        if (tid >= d) before += o;
      }
      before -= own;
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
    prefix = (prefix << 8) | digit;
    rem -= (int)above;
    __syncthreads();  // sel and hist are rewritten by the next pass
    if ((int)inbucket == rem || shift == 0) return prefix << shift;
  }
}

// Block sum / max over kScanThreads threads (four waves) through LDS.
__device__ __forceinline__ float block_sum4(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  const float s = (red[0] + red[1]) + (red[2] + red[3]);
  __syncthreads();
  return s;
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
  __shared__ uint32_t hist[256], sel[4];
  __shared__ float red[4];
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
  s = block_sum4(s, red);
  t = block_sum4(t, red);
  u = block_sum4(u, red);
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
  const uint64_t T = want < n ? select_threshold<kScanThreads, kScanItems>(key, want, hist, sel) : 1;
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

__global__ __launch_bounds__(kFinishThreads) void dgap_finish_kernel(DgapArgs a) {
  __shared__ uint32_t hist[256], sel[4];
  __shared__ uint64_t win[kDgapMaxK], skey[kDgapMaxK];
  __shared__ float stat[8];      // lse, H, sum p^2, r
  __shared__ float phi[kDgapFeatures];
  __shared__ float vsorted[kDgapMaxK];
  const int row = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int K = a.k, ncand = a.nchunk * K;
  float* z = a.logits + (size_t)row * a.vocab;

  // log-sum-exp, entropy and concentration from the chunk sums (wave 0)
  if (wv == 0) {
    const float* st = a.ws_stats + (size_t)row * a.nchunk * 4;
    float M = -__builtin_inff();
    for (int c = lane; c < a.nchunk; c += 64) M = fmaxf(M, st[4 * c]);
    M = wave_max(M);
    float S = 0.f;
    for (int c = lane; c < a.nchunk; c += 64) S += expf(st[4 * c] - M) * st[4 * c + 1];
    S = wave_sum(S);
    const float lse = M + logf(S);
    // H = sum_i p_i (lse - z_i) = sum_chunks e^(m-lse) ((lse - m) s + sum_i e_i (m - z_i)),
    // every term non-negative
    float h = 0.f, p2 = 0.f;
    for (int c = lane; c < a.nchunk; c += 64) {
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
  uint64_t key[kFinishItems];
  const uint64_t* cand = a.ws_cand + (size_t)row * ncand;
#pragma unroll
  for (int j = 0; j < kFinishItems; ++j) {
    const int i = j * kFinishThreads + tid;
    key[j] = i < ncand ? cand[i] : 0;
  }
  const uint64_t T = select_threshold<kFinishThreads, kFinishItems>(key, K, hist, sel);
  if (tid == 0) sel[3] = 0;
  __syncthreads();
#pragma unroll
  for (int j = 0; j < kFinishItems; ++j)
    if (key[j] != 0 && key[j] >= T) {
      const uint32_t slot = atomicAdd(&sel[3], 1u);
      if (slot < (uint32_t)K) win[slot] = key[j];  // exactly K keys pass
    }
  __syncthreads();
  if (tid < K) {
    const uint64_t mine = win[tid];
    int rank = 0;
    for (int j = 0; j < K; ++j) rank += win[j] > mine;
    skey[rank] = mine;
    vsorted[rank] = key_value(mine);
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
    if (lane < a.hidden_det) {
      float acc = a.det_b1[lane];
#pragma unroll
      for (int i = 0; i < kDgapFeatures; ++i) acc = fmaf(phi[i], a.det_w1[i * a.hidden_det + lane], acc);
      y = fmaxf(acc, 0.f) * a.det_w2[lane];
    }
    const float s = wave_sum(y) + a.det_b2;
    if (lane == 0) stat[3] = 1.f / (1.f + expf(-s));
  }
  __syncthreads();
  const float r = stat[3];
  const bool correct = r > a.tau;
  float* info = a.info ? a.info + (size_t)row * (kDgapInfoHead + 2 * K) : nullptr;

  if (correct) {
    // corrector: lane h is hidden unit h; the phi part of its input is the
    // same for every candidate
    float uh = 0.f, w2h = 0.f, wx[kDgapCandInputs];
    if (lane < a.hidden_corr) {
      uh = a.corr_b1[lane];
#pragma unroll
      for (int i = 0; i < kDgapFeatures; ++i)
        uh = fmaf(phi[i], a.corr_w1[(kDgapCandInputs + i) * a.hidden_corr + lane], uh);
      w2h = a.corr_w2[lane];
#pragma unroll
      for (int i = 0; i < kDgapCandInputs; ++i) wx[i] = a.corr_w1[i * a.hidden_corr + lane];
    } else {
#pragma unroll
      for (int i = 0; i < kDgapCandInputs; ++i) wx[i] = 0.f;
    }
    for (int k = wv; k < K; k += kFinishThreads / 64) {
      const float vk = vsorted[k];
      const float xi[kDgapCandInputs] = {vk - vsorted[0], vk - lse, (float)k / (float)(K - 1),
                                         k > 0 ? vsorted[k - 1] - vk : 0.f, k + 1 < K ? vk - vsorted[k + 1] : 0.f};
      float acc = uh;
#pragma unroll
      for (int i = 0; i < kDgapCandInputs; ++i) acc = fmaf(xi[i], wx[i], acc);
      const float d = wave_sum(fmaxf(acc, 0.f) * w2h) + a.corr_b2;
      if (lane == 0) {
        const uint32_t idx = key_index(skey[k]);
        if (idx < (uint32_t)a.vocab) z[idx] = vk + d;
        if (info) info[kDgapInfoHead + K + k] = d;
      }
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
  hipLaunchKernelGGL(dgap_finish_kernel, dim3(batch), dim3(kFinishThreads), 0, (hipStream_t)stream, a);
  return (int)hipGetLastError();
}

}  // namespace kvq
