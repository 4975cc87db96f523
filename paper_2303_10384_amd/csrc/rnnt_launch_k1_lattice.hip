// Kernel 1 instances writing the lattice form of the fused loss and forced alignment.
#include "rnnt_launch_k1.h"

namespace rnnt {

hipError_t launch_populate_lattice(rnnt_dtype_t dt, const PopulateParams& p, hipStream_t stream) {
  return k1::launch_k1_dtype<kK1Lattice>(dt, p, stream);
}

}  // namespace rnnt
