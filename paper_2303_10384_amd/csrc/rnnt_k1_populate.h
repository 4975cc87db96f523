// Kernel 1: row log-normaliser and gather of the blank / label log-probs.
//
// Populate (Section 2.2) selects every arc weight of the grid lattice (Fig. 1)
// from X = log_softmax(logits) by (time, unit_idx, label).  One pass over each
// valid logits row (t < T_b, u <= U_b) computes lse = ln sum_v exp z_v and
// emits only what the lattice needs:
//   lp_blank(t, u) = z[blank] - lse,  lp_label(t, u) = z[y_{u+1}] - lse
// (float64, formed from the exact input value), plus lse * log2(e) as float32
// for the gradient kernel.  Padding rows are never touched.
//
// Mapping: a block owns `rows_per_block` consecutive rows u of one (b, t)
// segment; a group of G lanes reads one row as aligned 16-byte chunks, NB
// chunks per lane per batch (G and NB are picked from V so that G*NB just
// covers a row).  All loads of a batch are issued unconditionally (chunk index
// clamped into the row) before any value is touched, and the elements outside
// the row are masked afterwards, so a row's loads are in flight together.  The
// group reduces max, then sum of exp in float32 per lane and float64 across
// lanes.  A row whose last chunk runs past the end of the tensor (only the
// tensor's last row can) takes an element-wise path.
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
  int32_t n_ublk;          // blocks per (b, t) segment
  int32_t rows_per_block;  // consecutive rows u per block
  RowInfo* rowinfo;        // row records (lse2 filled here) or null
  double* lp_blank;        // element (b,t,u) at b*sb + t*st + u*su (in doubles)
  double* lp_label;
  int64_t sb, st, su;
  double* lse_out;         // dense (B, T_max, U_max+1) or null
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

template <typename T, int G, int NB>
__global__ __launch_bounds__(256) void k1_populate(PopulateParams p) {
  constexpr int EPC = ElemTraits<T>::kPerChunk;
  constexpr int GROUPS = 256 / G;      // rows in flight per block
  constexpr int MAX_ROWS = GROUPS * 4; // rows_per_block set by the launcher
  const float kNegInf = -__builtin_inff();
  __shared__ int s_label[MAX_ROWS];

  const int seg = blockIdx.x / p.n_ublk;  // b * T_max + t
  const int ublk = blockIdx.x - seg * p.n_ublk;
  const int b = seg / p.T_max;
  const int t = seg - b * p.T_max;
  const int Tb = p.logit_lens[b];
  const int Ub = p.label_lens[b];
  if (Tb < 1 || Tb > p.T_max || Ub < 0 || Ub > p.U_max || t >= Tb) return;

  const int lg = threadIdx.x % G;  // lane inside the row group
  const int grp = threadIdx.x / G;
  const int u_begin = ublk * p.rows_per_block;
  const int u_end = min(u_begin + p.rows_per_block, Ub + 1);
  // the block's labels go through LDS, so no label load waits inside the row loop
  if (threadIdx.x < MAX_ROWS) {
    const int u = u_begin + threadIdx.x;
    s_label[threadIdx.x] = (u < Ub) ? p.labels[static_cast<int64_t>(b) * p.U_max + u] : kNoLabel;
  }
  __syncthreads();

  const T* __restrict__ base = static_cast<const T*>(p.logits);
  const uint4* __restrict__ cbase = reinterpret_cast<const uint4*>(base);
  const int64_t full_chunks = p.n_elem / EPC;

  for (int u = u_begin + grp; u < u_end; u += GROUPS) {
    const int64_t row = static_cast<int64_t>(seg) * (p.U_max + 1) + u;
    const int64_t e0 = row * p.V;
    const int64_t c0 = e0 / EPC;
    const int mis = static_cast<int>(e0 - c0 * EPC);
    const int nch = (mis + p.V + EPC - 1) / EPC;
    const int y = s_label[u - u_begin];
    const bool y_ok = (y >= 0 && y < p.V);
    // z[blank], z[y]: the same address in every lane of the group (one request,
    // the line the row's chunk loads bring in), issued ahead of them
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
      const int64_t li = static_cast<int64_t>(b) * p.sb + static_cast<int64_t>(t) * p.st +
                         static_cast<int64_t>(u) * p.su;
      p.lp_blank[li] = static_cast<double>(zb) - lse;
      double lpl = -__builtin_inf();
      if (u < Ub) lpl = y_ok ? static_cast<double>(zy) - lse : __builtin_nan("");
      p.lp_label[li] = lpl;
      if (p.rowinfo) p.rowinfo[row].lse2 = static_cast<float>(lse * kLog2eD);
      if (p.lse_out) p.lse_out[row] = lse;
    }
  }
}

}  // namespace rnnt
