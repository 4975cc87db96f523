// Kernel 1: row log-normaliser and gather of the blank / label log-probs.
//
// Populate (Section 2.2) selects every arc weight of the grid lattice (Fig. 1)
// from X = log_softmax(logits) by (time, unit_idx, label).  One pass over each
// valid logits row (t < T_b, u <= U_b) computes lse = ln sum_v exp z_v and
// emits only what the lattice needs, formed in float64 from the exact input:
//   lp_blank(t, u) = z[blank] - lse,  lp_label(t, u) = z[y_{u+1}] - lse.
// Padding rows are never touched.
//
// Two output forms:
//  * LATTICE (the fused loss): arc weights in log2 units, stored as
//    {lp_blank, lp_label} pairs by anti-diagonal (cell (t, u) of utterance b at
//    (b*(T_max+U_max) + t+u)*(U_max+1) + u), where the lattice kernel reads a
//    diagonal as one contiguous run; absent arcs (the label arc of the top row,
//    the blank arcs of the last frame below the top row) carry kNoArc; plus
//    lse * log2(e) as float32 at the same index.
//  * dense natural-log lse / lp_blank / lp_label, (B, T_max, U_max+1) float64
//    (the populate step on its own).
//
// Mapping: a block owns up to `rows_per_block` consecutive units u of one
// anti-diagonal d of one utterance, so the lattice-form writes of a block are
// one contiguous run; a group of G lanes reads one row as aligned 16-byte
// chunks, NB chunks per lane per batch (G, NB picked from V so that G*NB just
// covers a row).  All loads of a batch are issued unconditionally (chunk index
// clamped into the row) before any value is touched, and elements outside the
// row are masked afterwards.  The group reduces max, then sum of exp in
// float32 per lane and float64 across lanes.  A row whose last chunk runs past
// the end of the tensor (only the tensor's last row can) reads element-wise.
#pragma once

#include "rnnt_device.h"

namespace rnnt {

struct PopulateParams {
  const void* logits;
  int32_t B, T_max, U_max, V, blank;
  const int32_t* labels;
  const int32_t* logit_lens;
  const int32_t* label_lens;
  int64_t n_elem;          // B * T_max * (U_max+1) * V
  int32_t n_ublk;          // blocks per anti-diagonal
  int32_t rows_per_block;  // consecutive units u per block
  // lattice form
  double2* lp2;            // (B, T_max+U_max, U_max+1) {lp_blank, lp_label} * log2(e)
  float* lse2;             // same index: lse * log2(e)
  // dense form
  double* lse_out;         // (B, T_max, U_max+1) or null
  double* lp_blank_out;
  double* lp_label_out;
};

// (max, sum of exp) of one batch of register-held values, merged into the
// lane's running pair.
template <int N>
__device__ __forceinline__ void merge_batch(const float (&x)[N], float& mloc, float& sloc) {
  const float kNegInf = -__builtin_inff();
  float bm = kNegInf;
#pragma unroll
  for (int i = 0; i < N; ++i) bm = fmaxf(bm, x[i]);
  const float mn = fmaxf(mloc, bm);
  const float sh = (mn == kNegInf) ? 0.f : mn;
  float acc = 0.f;
#pragma unroll
  for (int i = 0; i < N; ++i) acc += fast_exp2((x[i] - sh) * kLog2eF);
  sloc = (mloc == kNegInf) ? acc : fmaf(sloc, fast_exp2((mloc - sh) * kLog2eF), acc);
  mloc = mn;
}

__device__ __forceinline__ double clamp_no_arc(double x) { return x < kNoArc ? kNoArc : x; }  // NaN stays NaN

template <typename T, int G, int NB, bool LATTICE>
__global__ __launch_bounds__(256) void k1_populate(PopulateParams p) {
  constexpr int EPC = ElemTraits<T>::kPerChunk;
  constexpr int GROUPS = 256 / G;      // rows in flight per block
  constexpr int MAX_ROWS = GROUPS * 4; // rows_per_block set by the launcher
  const float kNegInf = -__builtin_inff();
  __shared__ int s_label[MAX_ROWS];

  const int ND = p.T_max + p.U_max;  // anti-diagonals per utterance
  const int diag = blockIdx.x / p.n_ublk;  // b * ND + d
  const int ublk = blockIdx.x - diag * p.n_ublk;
  const int b = diag / ND;
  const int d = diag - b * ND;
  const int Tb = p.logit_lens[b];
  const int Ub = p.label_lens[b];
  if (Tb < 1 || Tb > p.T_max || Ub < 0 || Ub > p.U_max) return;
  const int u_first = ublk * p.rows_per_block;
  const int u_lo = max(u_first, d - (Tb - 1));           // t = d - u <= T_b - 1
  const int u_hi = min(u_first + p.rows_per_block, min(d, Ub) + 1);
  if (u_lo >= u_hi) return;

  const int lg = threadIdx.x % G;  // lane inside the row group
  const int grp = threadIdx.x / G;
  // the block's labels go through LDS, so no label load waits inside the row loop
  if (threadIdx.x < MAX_ROWS) {
    const int u = u_first + threadIdx.x;
    s_label[threadIdx.x] = (u < Ub) ? p.labels[static_cast<int64_t>(b) * p.U_max + u] : kNoLabel;
  }
  __syncthreads();

  const T* __restrict__ base = static_cast<const T*>(p.logits);
  const uint4* __restrict__ cbase = reinterpret_cast<const uint4*>(base);
  const int64_t full_chunks = p.n_elem / EPC;

  for (int u = u_first + grp; u < u_hi; u += GROUPS) {
    if (u < u_lo) continue;  // group-uniform
    const int t = d - u;
    const int64_t row = (static_cast<int64_t>(b) * p.T_max + t) * (p.U_max + 1) + u;
    const int64_t e0 = row * p.V;
    const int64_t c0 = e0 / EPC;
    const int mis = static_cast<int>(e0 - c0 * EPC);
    const int nch = (mis + p.V + EPC - 1) / EPC;
    const int y = s_label[u - u_first];
    const bool y_ok = (y >= 0 && y < p.V);
    // z[blank], z[y]: the same address in every lane of the group (one request,
    // a line the row's chunk loads bring in anyway), issued ahead of them
    const float zb = ElemTraits<T>::load1(base + e0 + p.blank);
    const float zy = ElemTraits<T>::load1(base + e0 + (y_ok ? y : 0));

    float mloc = kNegInf, sloc = 0.f;
    if (c0 + nch <= full_chunks) {
      for (int kb = 0; kb < nch; kb += G * NB) {
        uint4 raw[NB];
#pragma unroll
        for (int q = 0; q < NB; ++q) {
          const int k = min(kb + q * G + lg, nch - 1);
          raw[q] = cbase[c0 + k];
        }
        float x[NB * EPC];
#pragma unroll
        for (int q = 0; q < NB; ++q) {
          float f[EPC];
          ElemTraits<T>::unpack(raw[q], f);
          const int k = kb + q * G + lg;
#pragma unroll
          for (int j = 0; j < EPC; ++j) {
            const int v = k * EPC + j - mis;
            x[q * EPC + j] = (k < nch && v >= 0 && v < p.V) ? f[j] : kNegInf;
          }
        }
        merge_batch<NB * EPC>(x, mloc, sloc);
      }
    } else {
      // last row of the tensor, whose final chunk is partial: element loads
      for (int k = lg; k < nch; k += G) {
        float x[EPC];
#pragma unroll
        for (int j = 0; j < EPC; ++j) {
          const int v = k * EPC + j - mis;
          x[j] = (v >= 0 && v < p.V) ? ElemTraits<T>::load1(base + e0 + v) : kNegInf;
        }
        merge_batch<EPC>(x, mloc, sloc);
      }
    }

    // group max, then every lane's partial sum rescaled to it and summed in float64
    float mg = mloc;
#pragma unroll
    for (int off = G / 2; off > 0; off >>= 1) mg = fmaxf(mg, __shfl_xor(mg, off, G));
    const float scale = (mloc == kNegInf) ? 0.f : fast_exp2((mloc - mg) * kLog2eF);
    double sd = static_cast<double>(sloc * scale);
#pragma unroll
    for (int off = G / 2; off > 0; off >>= 1) sd += __shfl_xor(sd, off, G);

    if (lg == 0) {
      const double lse = static_cast<double>(mg) + log(sd);
      const double lpb = static_cast<double>(zb) - lse;
      const double lpl = (u < Ub) ? (y_ok ? static_cast<double>(zy) - lse : __builtin_nan("")) : -__builtin_inf();
      if (LATTICE) {
        const int64_t sc = static_cast<int64_t>(diag) * (p.U_max + 1) + u;
        const bool blank_arc = (t < Tb - 1) || (u == Ub);  // absent: last frame below the top row
        double2 w;
        w.x = blank_arc ? clamp_no_arc(lpb * kLog2eD) : kNoArc;
        w.y = (u < Ub) ? clamp_no_arc(lpl * kLog2eD) : kNoArc;
        p.lp2[sc] = w;
        p.lse2[sc] = static_cast<float>(lse * kLog2eD);
      } else {
        if (p.lse_out) p.lse_out[row] = lse;
        p.lp_blank_out[row] = lpb;
        p.lp_label_out[row] = lpl;
      }
    }
  }
}

}  // namespace rnnt
