// Host stand-ins for the HIP runtime calls and kernel launchers of the
// library (see hip/hip_runtime.h in this directory).  Copies are memcpy on
// host buffers, so every offset the host code computes into the arena, the
// workspace or an export buffer is checked by AddressSanitizer; launches
// only record that they happened.
#include <hip/hip_runtime.h>

#include <cstdlib>
#include <cstring>

#include "kvq_internal.h"

int g_launches = 0;

hipError_t hipGetDevice(int* dev) {
  *dev = 0;
  return hipSuccess;
}
hipError_t hipDeviceGetAttribute(int* value, hipDeviceAttribute_t, int) {
  *value = 256;
  return hipSuccess;
}
const char* hipGetErrorString(hipError_t) { return "stub"; }
hipError_t hipMemcpy(void* dst, const void* src, size_t bytes, hipMemcpyKind) {
  std::memmove(dst, src, bytes);
  return hipSuccess;
}
hipError_t hipMemcpyAsync(void* dst, const void* src, size_t bytes, hipMemcpyKind, hipStream_t) {
  std::memmove(dst, src, bytes);
  return hipSuccess;
}
hipError_t hipStreamSynchronize(hipStream_t) { return hipSuccess; }

namespace kvq {
int launch_append(const AppendArgs&, int, int, void*) { return ++g_launches, 0; }
int launch_table_set(const TableSet& t, void*) {
  // the table lives in the arena: write it as the kernel would
  for (int i = 0; i < t.n; ++i) t.table[t.idx[i]] = t.val[i];
  return ++g_launches, 0;
}
int launch_word_reset(const WordReset& r, void*) {
  for (int i = 0; i < r.n; ++i) std::memset(r.arena + r.off[i], 0, 4);
  return ++g_launches, 0;
}
int launch_decode(const DecodeArgs&, int, int, int, void*) { return ++g_launches, 0; }
int launch_decode_matrix(const DecodeArgs&, int, int, int, void*) { return ++g_launches, 0; }
int launch_chunk_matrix(const DecodeArgs&, int, int, int, void*) { return ++g_launches, 0; }
int launch_export(const ExportArgs&, void*) { return ++g_launches, 0; }
int launch_merge(const MergeArgs&, void*) { return ++g_launches, 0; }
int launch_dgap(const DgapArgs&, int, void*) { return ++g_launches, 0; }
int launch_dequant(const DequantArgs&, void*) { return ++g_launches, 0; }
int launch_fill_zero(void* dst, size_t words, void*) {
  std::memset(dst, 0, words * 4);
  return ++g_launches, 0;
}
int launch_read_probe(const void*, size_t, uint32_t*, void*) { return ++g_launches, 0; }
int read_probe_blocks() { return 2048; }
int scratch_workspace(void** ptr) {
  static void* buf = nullptr;
  if (!buf) buf = std::calloc(1, kScratchBytes);
  *ptr = buf;
  return 0;
}
}  // namespace kvq
