// Sweeps and posteriors on given dense float64 lattice weights.
#include "rnnt_launch_k2.h"

namespace rnnt {

hipError_t launch_lattice_dense(int variant, const LatticeParams& p, hipStream_t stream) {
  return k2::launch_k2<kScores, true>(variant, p, stream);
}

hipError_t launch_posteriors_dense(const PostParams& p, hipStream_t stream) { return k2::launch_k2b<true>(p, stream); }

}  // namespace rnnt
