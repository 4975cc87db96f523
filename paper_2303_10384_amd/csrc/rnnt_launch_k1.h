// Launch templates of kernel 1 (row log-normaliser and gather): row-group shape
// from V, blocking of the diagonals, and the template instance for the dtype.
// Included by the three units that instantiate one output form each
// (rnnt_launch_k1_lattice.hip, rnnt_launch_k1_rows.hip, rnnt_launch_k1_dense.hip).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "rnnt_launch.h"

namespace rnnt {
namespace k1 {
namespace {  // each including unit keeps its own copy

// ---- kernel 1 ---------------------------------------------------------------

// Lanes per row G and interior chunks per lane NB: the smallest G*NB that
// covers a row's interior chunks (at most V / EPC of them) with NB <= 5; rows
// with more take the batched path (G = 64, NB = 5).
struct K1Shape {
  int G, NB;
  bool fast;
};

template <typename T>
K1Shape k1_shape(int V) {
  constexpr int EPC = ElemTraits<T>::kPerChunk;
  const int interior = V / EPC;
  K1Shape best{64, 5, false};
  int best_slots = 1 << 30;
  // ties go to the larger G (fewer chunks per lane; measured faster on 16-bit
  // rows of 1025, where G = 32 x NB = 4 and G = 64 x NB = 2 tie)
  for (int g : {8, 16, 32, 64}) {
    for (int nb = 1; nb <= 5; ++nb) {
      const int slots = g * nb;
      if (slots >= interior && slots <= best_slots) {
        best = K1Shape{g, nb, true};
        best_slots = slots;
      }
    }
  }
  return best;
}

// one block per frame of an utterance, split into the fewest blocks of at most 32
// units for float32 rows and kMaxRowsPerBlock units for 16-bit ones, of equal size
// up to one unit (81 units: 27 + 27 + 27, not 32 + 32 + 17)
void k1_blocking(PopulateParams& p, int elem_bytes) {
  const int cap = elem_bytes == 4 ? 32 : kMaxRowsPerBlock;
  const int U1 = p.U_max + 1;
  p.n_ublk = (U1 + cap - 1) / cap;
  p.rows_per_block = (U1 + p.n_ublk - 1) / p.n_ublk;
}

template <typename T, int G, int NB, int OUT, bool FAST>
hipError_t launch_k1_g(PopulateParams p, hipStream_t stream) {
  k1_blocking(p, static_cast<int>(sizeof(T)));
  const int64_t blocks = static_cast<int64_t>(p.B) * p.T_max * p.n_ublk;
  const int64_t runs = (blocks + kXcdRun - 1) / kXcdRun;  // whole rounds of the XCD-major numbering
  const int64_t grid = (runs + kXcds - 1) / kXcds * kXcds * kXcdRun;
  if (grid > 0x7fffffffLL) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL((k1_populate<T, G, NB, OUT, FAST>), dim3(static_cast<uint32_t>(grid)), dim3(256), 0,
                     stream, p);
  return hipGetLastError();
}

template <typename T, int G, int OUT>
hipError_t launch_k1_nb(int nb, const PopulateParams& p, hipStream_t stream) {
  switch (nb) {
    case 1: return launch_k1_g<T, G, 1, OUT, true>(p, stream);
    case 2: return launch_k1_g<T, G, 2, OUT, true>(p, stream);
    case 3: return launch_k1_g<T, G, 3, OUT, true>(p, stream);
    case 4: return launch_k1_g<T, G, 4, OUT, true>(p, stream);
    default: return launch_k1_g<T, G, 5, OUT, true>(p, stream);
  }
}

// A block's rows are consecutive; the fast path addresses them through one
// buffer resource with 32-bit offsets.
bool k1_span_fits(PopulateParams p, int elem_bytes) {
  k1_blocking(p, elem_bytes);
  return static_cast<int64_t>(p.rows_per_block) * p.V * elem_bytes + 64 < 0x7fffffffLL;
}

template <typename T, int OUT>
hipError_t launch_k1(const PopulateParams& p, hipStream_t stream) {
  const K1Shape ks = k1_shape<T>(p.V);
  if (!ks.fast || !k1_span_fits(p, static_cast<int>(sizeof(T)))) return launch_k1_g<T, 64, 5, OUT, false>(p, stream);
  switch (ks.G) {
    case 8: return launch_k1_nb<T, 8, OUT>(ks.NB, p, stream);
    case 16: return launch_k1_nb<T, 16, OUT>(ks.NB, p, stream);
    case 32: return launch_k1_nb<T, 32, OUT>(ks.NB, p, stream);
    default: return launch_k1_nb<T, 64, OUT>(ks.NB, p, stream);
  }
}

template <int OUT>
hipError_t launch_k1_dtype(rnnt_dtype_t dt, const PopulateParams& p, hipStream_t stream) {
  switch (dt) {
    case RNNT_DTYPE_F32: return launch_k1<float, OUT>(p, stream);
    case RNNT_DTYPE_BF16: return launch_k1<bf16_t, OUT>(p, stream);
    default: return launch_k1<f16_t, OUT>(p, stream);
  }
}

}  // namespace
}  // namespace k1
}  // namespace rnnt
