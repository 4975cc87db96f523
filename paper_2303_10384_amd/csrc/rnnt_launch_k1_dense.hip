// Kernel 1 instances writing the dense natural-log form of the populate step on its own.
#include "rnnt_launch_k1.h"

namespace rnnt {

hipError_t launch_populate_dense(rnnt_dtype_t dt, const PopulateParams& p, hipStream_t stream) {
  return k1::launch_k1_dtype<kK1Dense>(dt, p, stream);
}

}  // namespace rnnt
