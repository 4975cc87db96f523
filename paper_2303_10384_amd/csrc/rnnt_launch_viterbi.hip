// Forced-alignment sweep and backtrace.
#include "rnnt_launch_k2.h"

namespace rnnt {

hipError_t launch_viterbi(int variant, const ViterbiParams& p, hipStream_t stream) {
  return k2::launch_k2v(variant, p, stream);
}

}  // namespace rnnt
