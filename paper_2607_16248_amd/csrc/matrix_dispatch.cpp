// Launch of the matrix-core decode kernels: the bit class picks the object
// (decode_mfma.hip, compiled once per class) whose kernels run.
#include <hip/hip_runtime.h>

#include "kvq_internal.h"

namespace kvq {

int launch_decode_matrix(const DecodeArgs& a, int bk, int bv, int gq, void* stream) {
  if (a.total_wg <= 0) return 0;
  if (bk == 1 && bv == 1) return launch_matrix_class<1, 1>(a, gq, stream);
  if (bk == 1 && bv == 2) return launch_matrix_class<1, 2>(a, gq, stream);
  if (bk == 2 && bv == 1) return launch_matrix_class<2, 1>(a, gq, stream);
  if (bk == 2 && bv == 2) return launch_matrix_class<2, 2>(a, gq, stream);
  if (bk == 4 && bv == 4) return launch_matrix_class<4, 4>(a, gq, stream);
  if (bk == 4 && bv == 8) return launch_matrix_class<4, 8>(a, gq, stream);
  if (bk == 8 && bv == 4) return launch_matrix_class<8, 4>(a, gq, stream);
  if (bk == 8 && bv == 8) return launch_matrix_class<8, 8>(a, gq, stream);
  return (int)hipErrorInvalidValue;
}

}  // namespace kvq
