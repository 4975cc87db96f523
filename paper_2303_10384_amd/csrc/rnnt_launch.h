// Kernel launchers of the library, called by the entry points in rnnt_api.hip
// and defined in the rnnt_launch_*.hip units (several small units, so that a
// build compiles the template instances in parallel).  Each returns the
// launch's hipError_t.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "rnnt_mi355x.h"
#include "rnnt_device.h"
#include "rnnt_k1_populate.h"
#include "rnnt_k2_lattice.h"
#include "rnnt_k3_grad.h"
#include "rnnt_k2_viterbi.h"
#include "rnnt_arc_kernels.h"

namespace rnnt {

// kernel 1, one function per output form
hipError_t launch_populate_lattice(rnnt_dtype_t dt, const PopulateParams& p, hipStream_t stream);
hipError_t launch_populate_rows(rnnt_dtype_t dt, const PopulateParams& p, hipStream_t stream);
hipError_t launch_populate_dense(rnnt_dtype_t dt, const PopulateParams& p, hipStream_t stream);
// kernel 2: both sweeps storing scores, the forward sweep alone, both sweeps on dense weights
hipError_t launch_lattice_scores(int variant, const LatticeParams& p, hipStream_t stream);
hipError_t launch_lattice_loss_only(int variant, const LatticeParams& p, hipStream_t stream);
hipError_t launch_lattice_dense(int variant, const LatticeParams& p, hipStream_t stream);
// kernel 2b: row records, or dense float64 outputs
hipError_t launch_posteriors_rows(const PostParams& p, hipStream_t stream);
hipError_t launch_posteriors_dense(const PostParams& p, hipStream_t stream);
// forced alignment sweep and backtrace
hipError_t launch_viterbi(int variant, const ViterbiParams& p, hipStream_t stream);
// kernel 3
hipError_t launch_grad(rnnt_dtype_t dt, rnnt_dtype_t gdt, const GradParams& p, hipStream_t stream);
// arc-list lattices: sweep (ns wavefronts per block, dm slots per state in registers),
// arc weights, arc posteriors and row records over n_rows rows, rows with several labels
hipError_t launch_arc_sweep(int ns, int dm, const ArcSweepParams& p, hipStream_t stream);
hipError_t launch_arc_weights(rnnt_dtype_t dt, const ArcPopulateParams& p, hipStream_t stream);
hipError_t launch_arc_posteriors(const ArcRowParams& p, int64_t n_rows, hipStream_t stream);
hipError_t launch_arc_extra_rows(rnnt_dtype_t dt, rnnt_dtype_t gdt, const ArcExtraParams& p, int n,
                                 hipStream_t stream);

}  // namespace rnnt
