// Launches of kernel 3 (fused gradient) and of the arc-list lattice kernels.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "rnnt_launch.h"

namespace rnnt {
namespace {

// ---- kernel 3 ---------------------------------------------------------------

template <typename Tin, typename Tout>
hipError_t launch_k3(const GradParams& p, hipStream_t stream) {
  constexpr int EPC = ElemTraits<Tin>::kPerChunk;
  const int64_t chunks = (p.n_elem + EPC - 1) / EPC;
  const int64_t blocks = (chunks + kGradTileChunks<Tin> - 1) / kGradTileChunks<Tin>;
  if (blocks > 0x7fffffffLL) return hipErrorInvalidConfiguration;
  if (p.V < EPC)
    hipLaunchKernelGGL((k3_grad<Tin, Tout, true>), dim3(static_cast<uint32_t>(blocks)), dim3(kGradThreads<Tin>), 0,
                       stream, p);
  else if (p.V >= kWideMinV<Tin>)
    hipLaunchKernelGGL((k3_grad_wide<Tin, Tout>), dim3(static_cast<uint32_t>(blocks)), dim3(kGradThreads<Tin>), 0,
                       stream, p);
  else
    hipLaunchKernelGGL((k3_grad<Tin, Tout, false>), dim3(static_cast<uint32_t>(blocks)), dim3(kGradThreads<Tin>), 0,
                       stream, p);
  return hipGetLastError();
}

hipError_t launch_k3_dtype(rnnt_dtype_t dt, rnnt_dtype_t gdt, const GradParams& p, hipStream_t stream) {
  const bool f32_out = gdt == RNNT_DTYPE_F32;
  switch (dt) {
    case RNNT_DTYPE_F32: return launch_k3<float, float>(p, stream);
    case RNNT_DTYPE_BF16: return f32_out ? launch_k3<bf16_t, float>(p, stream) : launch_k3<bf16_t, bf16_t>(p, stream);
    default: return f32_out ? launch_k3<f16_t, float>(p, stream) : launch_k3<f16_t, f16_t>(p, stream);
  }
}

template <int NW, int DM>
hipError_t launch_sweep_t(const ArcSweepParams& p, hipStream_t stream) {
  hipLaunchKernelGGL((k_arc_sweep<NW, DM>), dim3(2 * p.B), dim3(64 * NW), 0, stream, p);
  return hipGetLastError();
}

template <int NS>
hipError_t launch_sweep_ns(int dm, const ArcSweepParams& p, hipStream_t stream) {
  switch (dm) {
    case 1: return launch_sweep_t<NS, 1>(p, stream);
    case 2: return launch_sweep_t<NS, 2>(p, stream);
    default: return launch_sweep_t<NS, 4>(p, stream);
  }
}

// one wavefront per chunk of 64 states of the plan's typical level, up to DM slots
// per state held in registers
hipError_t launch_sweep(int ns, int dm, const ArcSweepParams& p, hipStream_t stream) {
  switch (ns) {
    case 1: return launch_sweep_ns<1>(dm, p, stream);
    case 2: return launch_sweep_ns<2>(dm, p, stream);
    default: return launch_sweep_ns<4>(dm, p, stream);
  }
}

hipError_t launch_arc_populate(rnnt_dtype_t dt, const ArcPopulateParams& p, hipStream_t stream) {
  const int n = p.n_slots0 > p.n_slots1 ? p.n_slots0 : p.n_slots1;
  if (n == 0) return hipSuccess;
  const dim3 grid((n + 255) / 256);
  switch (dt) {
    case RNNT_DTYPE_F32: hipLaunchKernelGGL((k_arc_populate<float>), grid, dim3(256), 0, stream, p); break;
    case RNNT_DTYPE_BF16: hipLaunchKernelGGL((k_arc_populate<bf16_t>), grid, dim3(256), 0, stream, p); break;
    default: hipLaunchKernelGGL((k_arc_populate<f16_t>), grid, dim3(256), 0, stream, p); break;
  }
  return hipGetLastError();
}

template <typename Tin, typename Tout>
hipError_t launch_extra_rows_t(const ArcExtraParams& p, int n, hipStream_t stream) {
  hipLaunchKernelGGL((k_arc_extra_rows<Tin, Tout>), dim3(n), dim3(256), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_extra_rows(rnnt_dtype_t dt, rnnt_dtype_t gdt, const ArcExtraParams& p, int n, hipStream_t stream) {
  if (n == 0) return hipSuccess;
  const bool f32_out = gdt == RNNT_DTYPE_F32;
  switch (dt) {
    case RNNT_DTYPE_F32: return launch_extra_rows_t<float, float>(p, n, stream);
    case RNNT_DTYPE_BF16:
      return f32_out ? launch_extra_rows_t<bf16_t, float>(p, n, stream) : launch_extra_rows_t<bf16_t, bf16_t>(p, n, stream);
    default:
      return f32_out ? launch_extra_rows_t<f16_t, float>(p, n, stream) : launch_extra_rows_t<f16_t, f16_t>(p, n, stream);
  }
}

}  // namespace

hipError_t launch_grad(rnnt_dtype_t dt, rnnt_dtype_t gdt, const GradParams& p, hipStream_t stream) {
  return launch_k3_dtype(dt, gdt, p, stream);
}

hipError_t launch_arc_sweep(int ns, int dm, const ArcSweepParams& p, hipStream_t stream) {
  return launch_sweep(ns, dm, p, stream);
}

hipError_t launch_arc_weights(rnnt_dtype_t dt, const ArcPopulateParams& p, hipStream_t stream) {
  return launch_arc_populate(dt, p, stream);
}

hipError_t launch_arc_posteriors(const ArcRowParams& p, int64_t n_rows, hipStream_t stream) {
  constexpr int NT = 256;
  if (p.n_arcs > 0) {
    hipLaunchKernelGGL(k_arc_occ<NT>, dim3(static_cast<uint32_t>((p.n_arcs + NT - 1) / NT)), dim3(NT), 0, stream, p);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(k_arc_rows<NT>, dim3(static_cast<uint32_t>((n_rows + NT - 1) / NT)), dim3(NT), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_arc_extra_rows(rnnt_dtype_t dt, rnnt_dtype_t gdt, const ArcExtraParams& p, int n,
                                 hipStream_t stream) {
  return launch_extra_rows(dt, gdt, p, n, stream);
}

}  // namespace rnnt
