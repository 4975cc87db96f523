// Launch templates of the lattice sweeps (kernel 2), the arc posteriors (kernel
// 2b) and the forced-alignment sweep, by units per lane and lattice variant.
// Included by the units that instantiate them (rnnt_launch_k2_scores.hip,
// rnnt_launch_k2_loss.hip, rnnt_launch_k2_dense.hip, rnnt_launch_viterbi.hip).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "rnnt_launch.h"

namespace rnnt {
namespace k2 {
namespace {  // each including unit keeps its own copy

// ---- kernel 2 ---------------------------------------------------------------

template <int K, int VAR, int MODE, bool DENSE_IN, int NW = 1>
hipError_t launch_k2_k(const LatticeParams& p, hipStream_t stream) {
  constexpr int PF = (K >= 24) ? 1 : (K >= 16) ? 2 : (48 / K > 24 ? 24 : 48 / K);  // diagonals of weights in flight
  const int sweeps = (MODE == kLossOnly) ? 1 : 2;  // forward only, or forward and backward
  hipLaunchKernelGGL((k2_lattice<K, PF, VAR, MODE, DENSE_IN, NW>), dim3(p.B, sweeps), dim3(64 * NW), 0, stream, p);
  return hipGetLastError();
}

// Up to 256 units a sweep takes one unit per lane over as many wavefronts as it
// needs (the score rows keep the same 64 * units_per_lane columns); wider
// lattices take one wavefront with several units per lane.
#ifndef RNNT_K2_MULTI_WAVE
#define RNNT_K2_MULTI_WAVE 1
#endif
template <int VAR, int MODE, bool DENSE_IN>
hipError_t launch_k2_v(const LatticeParams& p, hipStream_t stream) {
  switch (units_per_lane(p.U_max + 1)) {
    case 1: return launch_k2_k<1, VAR, MODE, DENSE_IN>(p, stream);
#if RNNT_K2_MULTI_WAVE
    case 2: return launch_k2_k<1, VAR, MODE, DENSE_IN, 2>(p, stream);
    case 3: return launch_k2_k<1, VAR, MODE, DENSE_IN, 3>(p, stream);
    case 4: return launch_k2_k<1, VAR, MODE, DENSE_IN, 4>(p, stream);
#else
    case 2: return launch_k2_k<2, VAR, MODE, DENSE_IN>(p, stream);
    case 3: return launch_k2_k<3, VAR, MODE, DENSE_IN>(p, stream);
    case 4: return launch_k2_k<4, VAR, MODE, DENSE_IN>(p, stream);
#endif
    case 6: return launch_k2_k<6, VAR, MODE, DENSE_IN>(p, stream);
    case 8: return launch_k2_k<8, VAR, MODE, DENSE_IN>(p, stream);
    case 12: return launch_k2_k<12, VAR, MODE, DENSE_IN>(p, stream);
    case 16: return launch_k2_k<16, VAR, MODE, DENSE_IN>(p, stream);
    case 24: return launch_k2_k<24, VAR, MODE, DENSE_IN>(p, stream);
    default: return launch_k2_k<32, VAR, MODE, DENSE_IN>(p, stream);
  }
}

template <int MODE, bool DENSE_IN>
hipError_t launch_k2(int variant, const LatticeParams& p, hipStream_t stream) {
  switch (variant) {
    case RNNT_VARIANT_RNNT: return launch_k2_v<0, MODE, DENSE_IN>(p, stream);
    case RNNT_VARIANT_WRNNT: return launch_k2_v<1, MODE, DENSE_IN>(p, stream);
    default: return launch_k2_v<2, MODE, DENSE_IN>(p, stream);
  }
}

template <int K, int VAR, int NW = 1>
hipError_t launch_k2v_k(const ViterbiParams& p, hipStream_t stream) {
  constexpr int PF = (K >= 24) ? 1 : (K >= 16) ? 2 : (48 / K > 24 ? 24 : 48 / K);
  hipLaunchKernelGGL((k2_viterbi<K, PF, VAR, NW>), dim3(p.B), dim3(64 * NW), 0, stream, p);
  return hipGetLastError();
}

// the forced-alignment sweep splits over wavefronts as kernel 2 does (65 to 256 units)
template <int VAR>
hipError_t launch_k2v_v(const ViterbiParams& p, hipStream_t stream) {
  switch (units_per_lane(p.U_max + 1)) {
    case 1: return launch_k2v_k<1, VAR>(p, stream);
#if RNNT_K2_MULTI_WAVE
    case 2: return launch_k2v_k<1, VAR, 2>(p, stream);
    case 3: return launch_k2v_k<1, VAR, 3>(p, stream);
    case 4: return launch_k2v_k<1, VAR, 4>(p, stream);
#else
    case 2: return launch_k2v_k<2, VAR>(p, stream);
    case 3: return launch_k2v_k<3, VAR>(p, stream);
    case 4: return launch_k2v_k<4, VAR>(p, stream);
#endif
    case 6: return launch_k2v_k<6, VAR>(p, stream);
    case 8: return launch_k2v_k<8, VAR>(p, stream);
    case 12: return launch_k2v_k<12, VAR>(p, stream);
    case 16: return launch_k2v_k<16, VAR>(p, stream);
    case 24: return launch_k2v_k<24, VAR>(p, stream);
    default: return launch_k2v_k<32, VAR>(p, stream);
  }
}

inline hipError_t launch_k2v(int variant, const ViterbiParams& p, hipStream_t stream) {
  switch (variant) {
    case RNNT_VARIANT_RNNT: return launch_k2v_v<0>(p, stream);
    case RNNT_VARIANT_WRNNT: return launch_k2v_v<1>(p, stream);
    default: return launch_k2v_v<2>(p, stream);
  }
}

template <bool DENSE>
hipError_t launch_k2b(const PostParams& p, hipStream_t stream) {
  const int64_t blocks = static_cast<int64_t>(p.B) * ((p.T_max + kPostTileT - 1) / kPostTileT);
  if (blocks > 0x7fffffffLL) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL((k2b_posteriors<DENSE>), dim3(static_cast<uint32_t>(blocks)), dim3(kPostThreads), 0, stream, p);
  return hipGetLastError();
}

}  // namespace
}  // namespace k2
}  // namespace rnnt
