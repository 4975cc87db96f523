// Kernel 1 instances writing the rows form of the arc-list loss.
#include "rnnt_launch_k1.h"

namespace rnnt {

hipError_t launch_populate_rows(rnnt_dtype_t dt, const PopulateParams& p, hipStream_t stream) {
  return k1::launch_k1_dtype<kK1Rows>(dt, p, stream);
}

}  // namespace rnnt
