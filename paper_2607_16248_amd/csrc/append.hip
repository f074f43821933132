// Quantize-on-append for the packed low-bit KV cache (gfx950).
//
// One launch packs every key group that leaves the fp16 window and copies
// the remaining new tokens into the per-head fp16 ring.  The quantizer is
// asymmetric min-max with an fp16 scale rounded up and an fp16 zero-point
// equal to the group minimum; codes round half to even.  The paper names
// b-bit keys and values (Motivation, "Accuracy Loss under Aggressive KV
// Quantization") and asymmetric key/value formats (Related Work) but leaves
// the rule open; this is the rule the library defines in kvq.h.
//
// Exactness: x - z is exact in fp64, the fp64 quotient is correctly rounded
// (IEEE divide; this file is built with -ffp-contract=off and no fast-math)
// and rint() rounds half to even, so codes equal the exact rational
// round-half-even.  Off the decode hot path: a key group flushes once every
// key_group appended tokens.
#include <hip/hip_runtime.h>

#include "kvq_internal.h"
#include "kvq_layout.h"

namespace kvq {
namespace {

__device__ __forceinline__ double half_bits_to_double(uint16_t h) {
  return (double)__builtin_bit_cast(_Float16, h);
}

// Smallest fp16 (bit pattern) whose value is >= s, for 0 <= s <= 65504.
// Start from a rounded conversion and walk to the exact answer: positive fp16
// patterns increase with their value, and the conversion is within an ulp.
__device__ __forceinline__ bool half_ceil(double s, uint16_t& out) {
  if (!(s <= 65504.0) || !(s >= 0.0)) return false;
  if (s == 0.0) { out = 0; return true; }
  uint16_t b = __builtin_bit_cast(uint16_t, (_Float16)(float)s);
  while (half_bits_to_double(b) < s) ++b;
  while (b > 1 && half_bits_to_double((uint16_t)(b - 1)) >= s) --b;
  out = b;
  return true;
}

__device__ __forceinline__ void raise_range(uint8_t* arena) {
  *reinterpret_cast<volatile uint32_t*>(arena) = 4u;  // KVQ_ERR_RANGE
}

__device__ __forceinline__ const uint16_t* token_row(const AppendArgs& a, const AppendSeq& S,
                                                     const uint8_t* blk, uint32_t ring,
                                                     const uint16_t* in, int h, int p) {
  if (p < S.L_old) return reinterpret_cast<const uint16_t*>(blk + ring) + (size_t)(p % a.W) * kHeadDim;
  return in + (((size_t)S.seq * a.n_max + (p - S.L_old)) * a.hkv + h) * kHeadDim;
}

// Pack `rows` rows of 128 codes (LDS, row-major) at `bits` bits into dwords.
__device__ __forceinline__ void pack_rows(const uint8_t* codes, int rows, int bits, uint8_t* dst) {
  const int dw_per_row = 4 * bits, per_dw = 32 / bits;
  for (int k = threadIdx.x; k < rows * dw_per_row; k += blockDim.x) {
    const int i = k / dw_per_row, w = k % dw_per_row;
    uint32_t v = 0;
    for (int e = 0; e < per_dw; ++e) v |= (uint32_t)codes[i * kHeadDim + w * per_dw + e] << (e * bits);
    reinterpret_cast<uint32_t*>(dst + (size_t)i * 16 * bits)[w] = v;
  }
}

// Matrix layout (kvq_layout.h), key rows: each bit of a row dword comes from
// the channel and code bit key_bit_owner names.
__device__ __forceinline__ void pack_key_rows_matrix(const uint8_t* codes, int rows, int bits, uint8_t* dst) {
  const int dw_per_row = 4 * bits;
  for (int k = threadIdx.x; k < rows * dw_per_row; k += blockDim.x) {
    const int i = k / dw_per_row, w = k % dw_per_row;
    uint32_t v = 0;
    for (int q = 0; q < 32; ++q) {
      int c, p;
      key_bit_owner(w, q, bits, c, p);
      v |= (uint32_t)((codes[i * kHeadDim + c] >> p) & 1u) << q;
    }
    reinterpret_cast<uint32_t*>(dst + (size_t)i * 16 * bits)[w] = v;
  }
}

// Matrix layout, value codes: 32-token blocks of 512*b bytes in MFMA lane order.
__device__ __forceinline__ void pack_value_blocks_matrix(const uint8_t* codes, int rows, int bits, uint8_t* dst) {
  const int dw_per_block = 128 * bits;
  for (int k = threadIdx.x; k < (rows / 32) * dw_per_block; k += blockDim.x) {
    const int blk = k / dw_per_block, w = k % dw_per_block;
    uint32_t v = 0;
    for (int q = 0; q < 32; ++q) {
      int r, c, p;
      value_bit_owner(w, q, bits, r, c, p);
      v |= (uint32_t)((codes[(blk * 32 + r) * kHeadDim + c] >> p) & 1u) << q;
    }
    reinterpret_cast<uint32_t*>(dst + (size_t)blk * 512 * bits)[w] = v;
  }
}

__device__ void quantize_group(const AppendArgs& a, const AppendSeq& S, int h, int gi, int bk,
                               int bv, uint8_t* codes, uint32_t* vmax) {
  uint8_t* blk = a.arena + S.head0 + (uint64_t)h * a.head_stride;  // the fp16 ring's region
  const int gk = a.gk, j = S.Lq_old / gk + gi, p0 = j * gk;
  const int c = threadIdx.x;
  // the packed segment (head region or page) of the group, and the group's
  // first token and index in it
  int t0;
  uint8_t* seg = a.arena + packed_seg(a.pm, S.head0, a.head_stride, S.seq, h, p0, t0);
  const int jj = t0 / gk;

  // keys: thread c owns channel c of the group's gk tokens
  {
    double mn = __builtin_inf(), mx = -__builtin_inf();
    bool finite = true;
    for (int i = 0; i < gk; ++i) {
      const double v = half_bits_to_double(token_row(a, S, blk, a.tk, a.K, h, p0 + i)[c]);
      finite &= __builtin_isfinite(v);
      mn = v < mn ? v : mn;
      mx = v > mx ? v : mx;
    }
    if (mn == 0.0) mn = 0.0;  // +0 zero-point
    uint16_t sb = 0;
    const bool ok = finite && half_ceil((mx - mn) / (double)((1 << bk) - 1), sb);
    if (!ok) { raise_range(a.arena); sb = 0x7E00; }
    const double sv = half_bits_to_double(sb);
    for (int i = 0; i < gk; ++i) {
      const double v = half_bits_to_double(token_row(a, S, blk, a.tk, a.K, h, p0 + i)[c]);
      codes[i * kHeadDim + c] = (ok && sv != 0.0) ? (uint8_t)__builtin_rint((v - mn) / sv) : 0;
    }
    uint16_t* km = reinterpret_cast<uint16_t*>(seg + a.km) + (size_t)jj * 2 * kHeadDim;
    km[c] = sb;
    km[kHeadDim + c] = __builtin_bit_cast(uint16_t, (_Float16)mn);
  }
  __syncthreads();
  if (a.matrix)
    pack_key_rows_matrix(codes, gk, bk, seg + a.kc + (size_t)t0 * 16 * bk);
  else
    pack_rows(codes, gk, bk, seg + a.kc + (size_t)t0 * 16 * bk);
  __syncthreads();

  // values: one item per (token, value group); the largest value scale of
  // the group raises the head's bound (decode sizes its weight shift by it)
  if (threadIdx.x == 0) *vmax = 0u;
  __syncthreads();
  const int ng = kHeadDim / a.gv;
  for (int it = threadIdx.x; it < gk * ng; it += blockDim.x) {
    const int i = it / ng, g = it % ng;
    const uint16_t* row = token_row(a, S, blk, a.tv, a.V, h, p0 + i) + g * a.gv;
    double mn = __builtin_inf(), mx = -__builtin_inf();
    bool finite = true;
    for (int e = 0; e < a.gv; ++e) {
      const double v = half_bits_to_double(row[e]);
      finite &= __builtin_isfinite(v);
      mn = v < mn ? v : mn;
      mx = v > mx ? v : mx;
    }
    if (mn == 0.0) mn = 0.0;
    uint16_t sb = 0;
    const bool ok = finite && half_ceil((mx - mn) / (double)((1 << bv) - 1), sb);
    if (!ok) { raise_range(a.arena); sb = 0x7E00; }
    else atomicMax(vmax, (uint32_t)sb);  // positive fp16 patterns order like their values
    const double sv = half_bits_to_double(sb);
    for (int e = 0; e < a.gv; ++e) {
      const double v = half_bits_to_double(row[e]);
      codes[i * kHeadDim + g * a.gv + e] = (ok && sv != 0.0) ? (uint8_t)__builtin_rint((v - mn) / sv) : 0;
    }
    const uint32_t zb = __builtin_bit_cast(uint16_t, (_Float16)mn);
    if (a.matrix) {
      uint8_t* vmb = seg + a.vm + (size_t)((t0 + i) / 32) * 128 * ng;
      const int r = (t0 + i) % 32;
      *reinterpret_cast<uint16_t*>(vmb + value_meta_s(g, r)) = sb;
      *reinterpret_cast<uint16_t*>(vmb + value_meta_z(g, r, ng)) = (uint16_t)zb;
    } else {
      reinterpret_cast<uint32_t*>(seg + a.vm)[(size_t)(t0 + i) * ng + g] = (uint32_t)sb | (zb << 16);
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) atomicMax(reinterpret_cast<uint32_t*>(blk + a.vb), *vmax);
  if (a.matrix)
    pack_value_blocks_matrix(codes, gk, bv, seg + a.vc + (size_t)t0 * 16 * bv);
  else
    pack_rows(codes, gk, bv, seg + a.vc + (size_t)t0 * 16 * bv);
}

// Copy the new tokens that stay fp16 into the ring of head h.
__device__ void copy_ring(const AppendArgs& a, const AppendSeq& S, int h) {
  uint8_t* blk = a.arena + S.head0 + (uint64_t)h * a.head_stride;
  uint16_t* rk = reinterpret_cast<uint16_t*>(blk + a.tk);
  uint16_t* rv = reinterpret_cast<uint16_t*>(blk + a.tv);
  const int first = S.Lq_new > S.L_old ? S.Lq_new : S.L_old;
  const int c = threadIdx.x;
  for (int p = first; p < S.L_new; ++p) {
    const size_t src = (((size_t)S.seq * a.n_max + (p - S.L_old)) * a.hkv + h) * kHeadDim + c;
    rk[(size_t)(p % a.W) * kHeadDim + c] = a.K[src];
    rv[(size_t)(p % a.W) * kHeadDim + c] = a.V[src];
  }
}

__global__ __launch_bounds__(128) void append_kernel(AppendArgs a, int bk, int bv) {
  __shared__ uint8_t codes[128 * kHeadDim];
  __shared__ uint32_t vmax;
  const int wg = blockIdx.x;
  int si = 0;
  for (int i = 1; i < a.nseq; ++i) si = (a.seq[i].wg_begin <= wg) ? i : si;
  const AppendSeq& S = a.seq[si];
  const int local = wg - S.wg_begin;
  const int nquant = a.quantize ? S.n_quant * a.hkv : 0;
  if (local < nquant) {
    quantize_group(a, S, local / S.n_quant, local % S.n_quant, bk, bv, codes, &vmax);
  } else if (S.do_copy) {
    copy_ring(a, S, local - nquant);
  }
}

__global__ __launch_bounds__(256) void table_set_kernel(TableSet t) {
  for (int i = threadIdx.x; i < t.n; i += blockDim.x) t.table[t.idx[i]] = t.val[i];
}

__global__ __launch_bounds__(256) void word_reset_kernel(WordReset r) {
  for (int i = threadIdx.x; i < r.n; i += blockDim.x) *reinterpret_cast<uint32_t*>(r.arena + r.off[i]) = 0u;
}

__global__ __launch_bounds__(256) void fill_zero_kernel(uint32_t* p, size_t n) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    p[i] = 0u;
}

}  // namespace

int launch_append(const AppendArgs& a, int bk, int bv, void* stream) {
  if (a.total_wg <= 0) return 0;
  hipLaunchKernelGGL(append_kernel, dim3(a.total_wg), dim3(128), 0, (hipStream_t)stream, a, bk, bv);
  return (int)hipGetLastError();
}

int launch_table_set(const TableSet& t, void* stream) {
  if (t.n <= 0) return 0;
  hipLaunchKernelGGL(table_set_kernel, dim3(1), dim3(256), 0, (hipStream_t)stream, t);
  return (int)hipGetLastError();
}

int launch_word_reset(const WordReset& r, void* stream) {
  if (r.n <= 0) return 0;
  hipLaunchKernelGGL(word_reset_kernel, dim3(1), dim3(256), 0, (hipStream_t)stream, r);
  return (int)hipGetLastError();
}

int launch_fill_zero(void* dst, size_t words, void* stream) {
  if (words == 0) return 0;
  const unsigned blocks = (unsigned)((words + 255) / 256 < 1024 ? (words + 255) / 256 : 1024);
  hipLaunchKernelGGL(fill_zero_kernel, dim3(blocks), dim3(256), 0, (hipStream_t)stream,
                     (uint32_t*)dst, words);
  return (int)hipGetLastError();
}

}  // namespace kvq
