// Forward and backward sweeps of the fused loss with a gradient (both waves store
// their scores), and the posterior kernel writing row records.
#include "rnnt_launch_k2.h"

namespace rnnt {

hipError_t launch_lattice_scores(int variant, const LatticeParams& p, hipStream_t stream) {
  return k2::launch_k2<kScores, false>(variant, p, stream);
}

hipError_t launch_posteriors_rows(const PostParams& p, hipStream_t stream) { return k2::launch_k2b<false>(p, stream); }

}  // namespace rnnt
