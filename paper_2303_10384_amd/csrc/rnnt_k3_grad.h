// Kernel 3: fused gradient of sum_b loss_b with respect to the logits.
//
// The loss depends on logits row (t, u) only through the two arcs leaving node
// (t, u) (Fig. 1; the wild-card arcs of Fig. 4 carry no parameter), so with
// arc posteriors g_b, g_l and p = softmax(z):
//   d loss / d z_v = p_v (g_b + g_l) - g_b [v = blank] - g_l [v = y_{u+1}]
// The kernel streams the whole gradient tensor once: each 16-byte chunk is
// located in its row(s) by index arithmetic, rows flagged as zero rows
// (padding, bad utterances) are written as 0 without reading the logits, and
// every other chunk reads the logits once and writes the gradient once.
// p_v = exp2(z_v * log2(e) - lse2) with lse2 = lse * log2(e) from the row record.
#pragma once

#include "rnnt_device.h"

#ifndef RNNT_K3_NT_LOAD
#define RNNT_K3_NT_LOAD 1
#endif
#ifndef RNNT_K3_NT_STORE
#define RNNT_K3_NT_STORE 1
#endif

namespace rnnt {

constexpr bool kK3StreamLoads = RNNT_K3_NT_LOAD != 0;
constexpr bool kK3StreamStores = RNNT_K3_NT_STORE != 0;

struct GradParams {
  const void* logits;
  void* grad;
  const RowInfo* rowinfo;
  int64_t n_elem;  // B * T_max * (U_max+1) * V
  int64_t n_rows;  // B * T_max * (U_max+1)
  int32_t V, blank;
};

constexpr int kGradThreads = 256;
constexpr int kGradChunksPerThread = 4;
constexpr int kGradTileChunks = kGradThreads * kGradChunksPerThread;

__device__ __forceinline__ float grad_elem(float z, int v, const RowInfo& ri, int blank) {
  const float pr = fast_exp2(fmaf(z, kLog2eF, -ri.lse2));
  float g = pr * (ri.occ_blank + ri.occ_label);
  g = (v == blank) ? g - ri.occ_blank : g;
  g = (v == ri.label) ? g - ri.occ_label : g;
  return (ri.label == kZeroRow) ? 0.f : g;
}

// Gradient elements of one 16-byte input chunk, stored as Tout (one or two
// aligned 16-byte stores).
template <typename Tout, int EPC>
__device__ __forceinline__ void store_chunk(void* dst, int64_t e0, const float* out) {
  constexpr int PER = ElemTraits<Tout>::kPerChunk;
  static_assert(EPC % PER == 0, "input chunk must cover whole output chunks");
  uint4* d = reinterpret_cast<uint4*>(static_cast<Tout*>(dst) + e0);
#pragma unroll
  for (int i = 0; i < EPC / PER; ++i) store16<kK3StreamStores>(d + i, ElemTraits<Tout>::pack(out + i * PER));
}

// Tin: logits element type; Tout: gradient element type (Tin or float).
// SMALLV: V < elements per chunk, so one chunk may cover several rows.
template <typename Tin, typename Tout, bool SMALLV>
__global__ __launch_bounds__(kGradThreads) void k3_grad(GradParams p) {
  using T = Tin;
  constexpr int EPC = ElemTraits<T>::kPerChunk;
  const int64_t tile0 = static_cast<int64_t>(blockIdx.x) * kGradTileChunks;
  const int64_t e_tile = tile0 * EPC;
  const int64_t r_tile = e_tile / p.V;
  const uint32_t v_tile = static_cast<uint32_t>(e_tile - r_tile * p.V);
  const uint32_t uV = static_cast<uint32_t>(p.V);
  const uint4* __restrict__ src = static_cast<const uint4*>(p.logits);
  const T* __restrict__ src_e = static_cast<const T*>(p.logits);
  Tout* __restrict__ dst_e = static_cast<Tout*>(p.grad);

#pragma unroll
  for (int q = 0; q < kGradChunksPerThread; ++q) {
    const int cl = q * kGradThreads + static_cast<int>(threadIdx.x);
    const int64_t c = tile0 + cl;
    const int64_t e0 = c * EPC;
    if (e0 >= p.n_elem) break;
    const uint32_t off = v_tile + static_cast<uint32_t>(cl) * EPC;
    const uint32_t dr = off / uV;
    int64_t r = r_tile + dr;
    int v = static_cast<int>(off - dr * uV);
    const bool full = e0 + EPC <= p.n_elem;
    float out[EPC];

    if (!SMALLV) {
      const RowInfo ri0 = p.rowinfo[r];
      const bool split = v + EPC > p.V;
      RowInfo ri1 = ri0;
      if (split && r + 1 < p.n_rows) ri1 = p.rowinfo[r + 1];
      const bool zero0 = ri0.label == kZeroRow;
      const bool zero1 = ri1.label == kZeroRow;
      if (zero0 && (!split || zero1)) {
#pragma unroll
        for (int j = 0; j < EPC; ++j) out[j] = 0.f;
      } else {
        float f[EPC];
        if (full) {
          ElemTraits<T>::unpack(load16<kK3StreamLoads>(src + c), f);
        } else {
#pragma unroll
          for (int j = 0; j < EPC; ++j) f[j] = (e0 + j < p.n_elem) ? ElemTraits<T>::load1(src_e + e0 + j) : 0.f;
        }
#pragma unroll
        for (int j = 0; j < EPC; ++j) {
          const int vj = v + j;
          const bool second = vj >= p.V;
          out[j] = second ? grad_elem(f[j], vj - p.V, ri1, p.blank) : grad_elem(f[j], vj, ri0, p.blank);
        }
      }
    } else {
      float f[EPC];
      if (full) {
        ElemTraits<T>::unpack(load16<kK3StreamLoads>(src + c), f);
      } else {
#pragma unroll
        for (int j = 0; j < EPC; ++j) f[j] = (e0 + j < p.n_elem) ? ElemTraits<T>::load1(src_e + e0 + j) : 0.f;
      }
      RowInfo ri = p.rowinfo[r];
#pragma unroll
      for (int j = 0; j < EPC; ++j) {
        if (v >= p.V) {
          v -= p.V;
          ++r;
          if (r < p.n_rows) ri = p.rowinfo[r];
        }
        out[j] = grad_elem(f[j], v, ri, p.blank);
        ++v;
      }
    }
    if (full) {
      store_chunk<Tout, EPC>(p.grad, e0, out);
    } else {
#pragma unroll
      for (int j = 0; j < EPC; ++j)
        if (e0 + j < p.n_elem) ElemTraits<Tout>::store1(dst_e + e0 + j, out[j]);
    }
  }
}

}  // namespace rnnt
