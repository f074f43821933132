// Dequantization of a token range of one sequence, for checking (gfx950).
//
// A packed element becomes fma(code, s, z) in fp32: the exact z + code * s
// rounded once.  A tail element is its fp16 value.
#include <hip/hip_runtime.h>

#include "kvq_internal.h"
#include "kvq_layout.h"

namespace kvq {
namespace {

__device__ __forceinline__ float h2f(uint32_t bits16) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)bits16);
}

__device__ __forceinline__ uint32_t code_at(const uint8_t* row, int c, int bits) {
  const int bit = c * bits;
  return ((uint32_t)row[bit >> 3] >> (bit & 7)) & ((1u << bits) - 1u);
}

// Code of channel c from a matrix-layout key row / value block.
__device__ __forceinline__ uint32_t key_code_matrix(const uint8_t* row, int c, int bits) {
  uint32_t code = 0;
  for (int p = 0; p < bits; ++p) {
    const BitLoc b = key_bit(c, p, bits);
    code |= ((reinterpret_cast<const uint32_t*>(row)[b.word] >> b.bit) & 1u) << p;
  }
  return code;
}

__device__ __forceinline__ uint32_t value_code_matrix(const uint8_t* block, int r, int c, int bits) {
  uint32_t code = 0;
  for (int p = 0; p < bits; ++p) {
    const BitLoc b = value_bit(r, c, p, bits);
    code |= ((reinterpret_cast<const uint32_t*>(block)[b.word] >> b.bit) & 1u) << p;
  }
  return code;
}

__global__ __launch_bounds__(128) void dequant_kernel(DequantArgs a) {
  const int ti = blockIdx.x / a.hkv, h = blockIdx.x % a.hkv;
  const int p = a.tok0 + ti, c = threadIdx.x;
  const uint8_t* blk = a.arena + a.head0 + (uint64_t)h * a.head_stride;
  float kv, vv;
  if (p < a.Lq) {
    int q;  // p's position in its packed segment
    const uint8_t* seg = a.arena + packed_seg(a.pm, a.head0, a.head_stride, a.seq, h, p, q);
    const uint16_t* km = reinterpret_cast<const uint16_t*>(seg + a.km) + (size_t)(q / a.gk) * 2 * kHeadDim;
    const uint8_t* krow = seg + a.kc + (size_t)q * 16 * a.bk;
    const uint32_t kcode = a.matrix ? key_code_matrix(krow, c, a.bk) : code_at(krow, c, a.bk);
    kv = fmaf((float)kcode, h2f(km[c]), h2f(km[kHeadDim + c]));
    const int ng = kHeadDim / a.gv, g = c / a.gv;
    if (a.matrix) {
      const uint8_t* vblk = seg + a.vc + (size_t)(q / 32) * 512 * a.bv;
      const uint8_t* vmb = seg + a.vm + (size_t)(q / 32) * 128 * ng;
      const int r = q % 32;
      const uint32_t vcode = value_code_matrix(vblk, r, c, a.bv);
      vv = fmaf((float)vcode, h2f(*reinterpret_cast<const uint16_t*>(vmb + value_meta_s(g, r))),
                h2f(*reinterpret_cast<const uint16_t*>(vmb + value_meta_z(g, r, ng))));
    } else {
      const uint32_t meta = reinterpret_cast<const uint32_t*>(seg + a.vm)[(size_t)q * ng + g];
      vv = fmaf((float)code_at(seg + a.vc + (size_t)q * 16 * a.bv, c, a.bv), h2f(meta & 0xFFFF), h2f(meta >> 16));
    }
  } else {
    const size_t slot = (size_t)(p % a.W) * kHeadDim + c;
    kv = h2f(reinterpret_cast<const uint16_t*>(blk + a.tk)[slot]);
    vv = h2f(reinterpret_cast<const uint16_t*>(blk + a.tv)[slot]);
  }
  const size_t o = ((size_t)ti * a.hkv + h) * kHeadDim + c;
  a.K_out[o] = kv;
  a.V_out[o] = vv;
}

// One workgroup per 32-token block: codes into LDS, then canonical rows.
__global__ __launch_bounds__(256) void export_kernel(ExportArgs a) {
  __shared__ uint8_t kc[32 * kHeadDim], vc[32 * kHeadDim];
  const int b = blockIdx.x;
  const int ng = kHeadDim / a.gv;
  for (int idx = threadIdx.x; idx < 32 * kHeadDim; idx += blockDim.x) {
    const int r = idx / kHeadDim, c = idx % kHeadDim;
    kc[idx] = (uint8_t)key_code_matrix(a.blk + a.kc + (size_t)(32 * b + r) * 16 * a.bk, c, a.bk);
    vc[idx] = (uint8_t)value_code_matrix(a.blk + a.vc + (size_t)b * 512 * a.bv, r, c, a.bv);
  }
  __syncthreads();
  for (int k = threadIdx.x; k < 32 * 4 * a.bk; k += blockDim.x) {
    const int i = k / (4 * a.bk), w = k % (4 * a.bk), per = 32 / a.bk;
    uint32_t v = 0;
    for (int e = 0; e < per; ++e) v |= (uint32_t)kc[i * kHeadDim + w * per + e] << (e * a.bk);
    reinterpret_cast<uint32_t*>(a.kc_out + (size_t)(32 * b + i) * 16 * a.bk)[w] = v;
  }
  for (int k = threadIdx.x; k < 32 * 4 * a.bv; k += blockDim.x) {
    const int i = k / (4 * a.bv), w = k % (4 * a.bv), per = 32 / a.bv;
    uint32_t v = 0;
    for (int e = 0; e < per; ++e) v |= (uint32_t)vc[i * kHeadDim + w * per + e] << (e * a.bv);
    reinterpret_cast<uint32_t*>(a.vc_out + (size_t)(32 * b + i) * 16 * a.bv)[w] = v;
  }
  const uint8_t* vmb = a.blk + a.vm + (size_t)b * 128 * ng;
  for (int k = threadIdx.x; k < 32 * ng; k += blockDim.x) {
    const int r = k / ng, g = k % ng;
    const uint32_t sv = *reinterpret_cast<const uint16_t*>(vmb + value_meta_s(g, r));
    const uint32_t zv = *reinterpret_cast<const uint16_t*>(vmb + value_meta_z(g, r, ng));
    reinterpret_cast<uint32_t*>(a.vm_out)[(size_t)(32 * b + r) * ng + g] = sv | (zv << 16);
  }
}

}  // namespace

int launch_export(const ExportArgs& a, void* stream) {
  if (a.nblocks <= 0) return 0;
  hipLaunchKernelGGL(export_kernel, dim3(a.nblocks), dim3(256), 0, (hipStream_t)stream, a);
  return (int)hipGetLastError();
}

int launch_dequant(const DequantArgs& a, void* stream) {
  if (a.ntok <= 0) return 0;
  hipLaunchKernelGGL(dequant_kernel, dim3(a.ntok * a.hkv), dim3(kHeadDim), 0, (hipStream_t)stream, a);
  return (int)hipGetLastError();
}


// ---------------------------------------------------------------- read probe
//
// Streaming-read ceiling of the device: every thread reads 16-byte words in
// a grid-stride loop and folds them with XOR; one word per workgroup goes to
// `sink` so that the loads stay.  The decode kernels' algorithmic bytes are
// compared with this measured rate as well as with the nominal HBM peak.
namespace {
constexpr int kProbeBlocks = 2048;
__global__ __launch_bounds__(256) void read_probe_kernel(const uint4* __restrict__ src, size_t n, uint32_t* sink) {
  uint32_t acc = 0u;
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
    const uint4 v = src[i];
    acc ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  __shared__ uint32_t red[256];
  red[threadIdx.x] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t x = 0u;
    for (int t = 0; t < 256; ++t) x ^= red[t];
    sink[blockIdx.x] = x;
  }
}
}  // namespace

int read_probe_blocks() { return kProbeBlocks; }

int launch_read_probe(const void* src, size_t bytes, uint32_t* sink, void* stream) {
  if (bytes == 0) return 0;
  hipLaunchKernelGGL(read_probe_kernel, dim3(kProbeBlocks), dim3(256), 0, (hipStream_t)stream,
                     static_cast<const uint4*>(src), bytes / 16, sink);
  return (int)hipGetLastError();
}

}  // namespace kvq
