// Forward sweep of the fused loss without a gradient.
#include "rnnt_launch_k2.h"

namespace rnnt {

hipError_t launch_lattice_loss_only(int variant, const LatticeParams& p, hipStream_t stream) {
  return k2::launch_k2<kLossOnly, false>(variant, p, stream);
}

}  // namespace rnnt
