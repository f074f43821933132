// Host stand-ins for the HIP runtime calls and kernel launchers of the
// library (see hip/hip_runtime.h in this directory).  Copies are memcpy on
// host buffers, so every offset the host code computes into the arena, the
// workspace or an export buffer is checked by AddressSanitizer; launches
// only record that they happened.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "kvq_internal.h"

int g_launches = 0;
int g_row_plans = 0;  // chunk launches whose row groups were checked

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
}  // namespace kvq

// The row groups of a chunk launch, checked the way the kernels read them
// (query of row g = min(rg * qpr + row_x[g], nqry - 1), q row offset from the
// group's row 0, no record for spare rows): every q row read lies in the
// sequence's [nqry][Hq] block, every record row in [0, nqry * Hq), and every
// (query, head) of a kv head is written by exactly one row.
static void check_rows(const kvq::DecodeArgs& a, int rows) {
  if (a.nqry <= 1) return;
  auto bad = [&](const char* what, int rg, int g) {
    std::fprintf(stderr, "row check failed (%s): nqry %d qpr %d nrg %d gqh %d rows %d, group %d row %d\n", what,
                 a.nqry, a.qpr, a.nrg, a.gqh, rows, rg, g);
    std::abort();
  };
  if (rows < 1 || rows > 32 || a.qpr < 1 || a.qpr * a.gqh > rows || a.nrg != (a.nqry + a.qpr - 1) / a.qpr)
    bad("shape", -1, -1);
  std::vector<int> hits((size_t)a.nqry * a.gqh, 0);
  for (int h = 0; h < a.hkv; ++h)
    for (int rg = 0; rg < a.nrg; ++rg)
      for (int g = 0; g < rows; ++g) {
        const int j0 = rg * a.qpr + a.row_x[g];
        const int j = std::min(j0, a.nqry - 1);
        const int64_t qrow = (int64_t)rg * a.qpr * a.hq + h * a.gqh + a.row_off[g] - (int64_t)(j0 - j) * a.hq;
        if (qrow < 0 || qrow >= (int64_t)a.nqry * a.hq || qrow / a.hq != j) bad("q row", rg, g);
        const int64_t head = qrow % a.hq - (int64_t)h * a.gqh;
        if (head < 0 || head >= a.gqh) bad("q head", rg, g);
        if (j0 >= a.nqry) continue;  // spare: no record
        const int64_t rec = (int64_t)rg * a.qpr * a.hq + h * a.gqh + a.row_off[g];
        if (rec != qrow) bad("record row", rg, g);
        if (h == 0) ++hits[(size_t)j * a.gqh + head];
      }
  for (int v : hits)
    if (v != 1) bad("coverage", -1, -1);
  ++g_row_plans;
}

namespace kvq {
int launch_decode(const DecodeArgs& a, int, int, int rows, void*) { return check_rows(a, rows), ++g_launches, 0; }
int launch_decode_matrix(const DecodeArgs& a, int, int, int rows, void*) { return check_rows(a, rows), ++g_launches, 0; }
int launch_chunk_matrix(const DecodeArgs& a, int, int, int rows, void*) { return check_rows(a, rows), ++g_launches, 0; }
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
