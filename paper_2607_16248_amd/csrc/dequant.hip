// Dequantization of a token range of one sequence, for checking (gfx950).
//
// A packed element becomes fma(code, s, z) in fp32: the exact z + code * s
// rounded once.  A tail element is its fp16 value.
#include <hip/hip_runtime.h>

#include "kvq_internal.h"

namespace kvq {
namespace {

__device__ __forceinline__ float h2f(uint32_t bits16) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)bits16);
}

__device__ __forceinline__ uint32_t code_at(const uint8_t* row, int c, int bits) {
  const int bit = c * bits;
  return ((uint32_t)row[bit >> 3] >> (bit & 7)) & ((1u << bits) - 1u);
}

__global__ __launch_bounds__(128) void dequant_kernel(DequantArgs a) {
  const int ti = blockIdx.x / a.hkv, h = blockIdx.x % a.hkv;
  const int p = a.tok0 + ti, c = threadIdx.x;
  const uint8_t* blk = a.base + (uint64_t)h * a.head_stride;
  float kv, vv;
  if (p < a.Lq) {
    const uint16_t* km = reinterpret_cast<const uint16_t*>(blk + a.km) + (size_t)(p / a.gk) * 2 * kHeadDim;
    kv = fmaf((float)code_at(blk + a.kc + (size_t)p * 16 * a.bk, c, a.bk), h2f(km[c]), h2f(km[kHeadDim + c]));
    const int ng = kHeadDim / a.gv;
    const uint32_t meta = reinterpret_cast<const uint32_t*>(blk + a.vm)[(size_t)p * ng + c / a.gv];
    vv = fmaf((float)code_at(blk + a.vc + (size_t)p * 16 * a.bv, c, a.bv), h2f(meta & 0xFFFF), h2f(meta >> 16));
  } else {
    const size_t slot = (size_t)(p % a.W) * kHeadDim + c;
    kv = h2f(reinterpret_cast<const uint16_t*>(blk + a.tk)[slot]);
    vv = h2f(reinterpret_cast<const uint16_t*>(blk + a.tv)[slot]);
  }
  const size_t o = ((size_t)ti * a.hkv + h) * kHeadDim + c;
  a.K_out[o] = kv;
  a.V_out[o] = vv;
}

}  // namespace

int launch_dequant(const DequantArgs& a, void* stream) {
  if (a.ntok <= 0) return 0;
  hipLaunchKernelGGL(dequant_kernel, dim3(a.ntok * a.hkv), dim3(kHeadDim), 0, (hipStream_t)stream, a);
  return (int)hipGetLastError();
}

}  // namespace kvq
